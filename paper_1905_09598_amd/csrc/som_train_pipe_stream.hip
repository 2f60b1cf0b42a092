// Streamed-prototype instances of the pipelined training kernel of
// som_train_pipe.h.  They sit in a translation unit of their own because
// they are compiled without the structurizer option of the LDS-resident
// instances: in the streamed sweep it raises register pressure enough to
// cost more than the faster exchange polling it buys (see build.py).
#include "som_train_pipe.h"

namespace som {

PipeKernel pipe_stream_kernel(int m, int ks, int ns) {
    struct Entry {
        int m, ks, ns;
        PipeKernel fn;
    };
    // The shapes of the LDS-resident table whose sample registers leave
    // room for streamed rows (not KS = 7), on three sweepers; and one on
    // four sweepers (5-step blocks, rows of 512 float4: two slices each).
    static const Entry kStream[] = {
        {8, 1, 3, train_pipe_kernel<8, 1, false>}, {4, 1, 3, train_pipe_kernel<4, 1, false>},
        {4, 2, 3, train_pipe_kernel<4, 2, false>}, {4, 3, 3, train_pipe_kernel<4, 3, false>},
        {2, 3, 3, train_pipe_kernel<2, 3, false>}, {2, 4, 3, train_pipe_kernel<2, 4, false>},
        {5, 2, 4, train_pipe_kernel<5, 2, false, 0, 4>},
    };
    for (const Entry &e : kStream)
        if (e.m == m && e.ks == ks && e.ns == ns) return e.fn;
    return nullptr;
}

PipeKernel pipe_cols_kernel(int m, int rmax) {
    struct Entry {
        int m, rmax;
        PipeKernel fn;
    };
    static const Entry kCols[] = {
        {8, 10, train_pipe_kernel<8, 1, false, 10>},
    };
    for (const Entry &e : kCols)
        if (e.m == m && e.rmax == rmax) return e.fn;
    return nullptr;
}

}  // namespace som
