// Pipelined online-SOM training: the LDS-resident instances of the kernel
// in som_train_pipe.h, the launch planner and the launcher.
#include "som_train_pipe.h"

namespace som {
namespace {

using namespace dev;

typedef void (*DotsKernel)(TrainArgs, float *, int64_t);

struct PipeInstance {
    int m, ks;
    bool stream_ok;  // the streamed variant fits in registers
    PipeKernel lds;
};

template <int M, int KS, bool STREAM = true>
constexpr PipeInstance pipe_instance() {
    return PipeInstance{M, KS, STREAM, train_pipe_kernel<M, KS, true>};
}

// (M, KS): block length and float4 slices of 64 columns per sweeper (rows of
// up to 3 * 64 * KS float4).  The sample registers, 3 M KS float4 per lane,
// bound M * KS: the longer blocks (8 x 2, 6 x 3, 4 x 4) and KS = 7 stay out
// of scratch only in the LDS variant, which has no streamed row registers.
// The planner takes the cheapest shape for the row length: a longer block
// spreads the per-block hand-over between sweepers and controller over more
// steps, but its rows cost more per pass and its controller code (one
// unrolled exchange per step) grows.  The streamed kernels are listed in
// som_train_pipe_stream.hip.
const PipeInstance kPipe[] = {
    pipe_instance<8, 1>(),        pipe_instance<4, 1>(),        pipe_instance<8, 2, false>(),
    pipe_instance<4, 2>(),        pipe_instance<6, 3, false>(), pipe_instance<4, 3>(),
    pipe_instance<2, 3>(),        pipe_instance<4, 4, false>(), pipe_instance<2, 4>(),
    pipe_instance<2, 7, false>()};

const PipeInstance *pipe_for(int m, int ks) {
    for (const PipeInstance &p : kPipe)
        if (p.m == m && p.ks == ks) return &p;
    return nullptr;
}

size_t pipe_lds_bytes(int m, int rmax, int64_t P4, bool ldsw, bool cols = false,
                      int ns = kSweepers) {
    const size_t rp = (size_t)((rmax + 3) & ~3);
    size_t b = kPipeHeader + 2 * rp * ns * 2 * m * 4 + 2 * rp * (m + 1) * 4;
    b = (b + 15) & ~(size_t)15;
    b += rp * 16;
    // the column-walk sweep's discarded-write area, and 1 KB after the rows
    // that its LDS row loads read when it holds no rows in LDS
    if (cols) b += (size_t)kPipeDummy * 16 + 1024;
    if (ldsw) b += (size_t)rmax * P4 * 16;
    return b;
}

// Long-row (column-walk) instances: block length and row bound per
// workgroup (som_train_pipe_stream.hip).  Eight steps a block, the rows
// walked in two windows: on the 50 x 50 map at d = 10000, 8.51 us per step
// with four steps in one pass, 6.89 with six, 6.54 with six in two windows
// and 6.18 with eight (ten spill registers: 6.62; three windows reread the
// samples once more: 6.34 with twelve).
struct ColsInstance {
    int m, rmax;
};
const ColsInstance kCols[] = {{8, 10}};

// Streamed instances on four sweepers (block length, slices per sweeper):
// every SIMD sweeps, the controller shares the first one
// (som_train_pipe_stream.hip).  Five steps a block: on the 100 x 100 map at
// d = 2048, 5.04 us per step with four and 4.35 with five (prefetch two rows
// ahead); six steps spill registers and measured 4.71.
struct Wide {
    int m, ks;
};
const Wide kWide[] = {{5, 2}};

// The prepass kernel of the block's sample dot products, by block length.
DotsKernel block_dots_for(int m) {
    switch (m) {
    case 2: return block_dots_kernel<2>;
    case 4: return block_dots_kernel<4>;
    case 5: return block_dots_kernel<5>;
    case 6: return block_dots_kernel<6>;
    case 8: return block_dots_kernel<8>;
    default: return nullptr;
    }
}

// Measured exchange latency of the pipelined kernel (multi-poll, per-XCD
// replicated slots) by grid size, in microseconds.
double pipe_exchange_us(int g) {
    static const double gs[] = {1, 8, 64, 128, 256, 1024};
    static const double us[] = {0.1, 1.02, 1.03, 1.07, 1.18, 2.0};
    if (g <= 1) return us[0];
    for (int i = 1; i < 6; ++i)
        if (g <= gs[i]) {
            const double f = (log2((double)g) - log2(gs[i - 1])) / (log2(gs[i]) - log2(gs[i - 1]));
            return us[i - 1] + f * (us[i] - us[i - 1]);
        }
    return us[5];
}

}  // namespace

double plan_train_pipe(const TrainArgs &a, int num_cus, int max_lds, TrainPlan *plan) {
    const int64_t P4 = a.ld / 4;
    if (P4 % 64 != 0) return 1e300;
    const int nsl = (int)(P4 / 64);
    const int ks_need = (nsl + kSweepers - 1) / kSweepers;
    const int max_grid = a.N < num_cus ? a.N : num_cus;
    double best = 1e300;
    for (const PipeInstance &pi : kPipe) {
        if (pi.ks != ks_need || (a.block_m > 0 && pi.m != a.block_m) || a.sweepers == 4) continue;
        for (int v = 0; v < 2; ++v) {
            const bool ldsw = v == 0;  // LDS first: it wins ties
            if ((a.variant == 1 && !ldsw) || (a.variant == 2 && ldsw)) continue;
            if (!ldsw && !pi.stream_ok) continue;
            for (int g = 1;; g = (g * 2 > max_grid && g < max_grid) ? max_grid : g * 2) {
                const int gg = a.grid > 0 ? (a.grid < a.N ? a.grid : a.N) : g;
                const int rmax = (a.N + gg - 1) / gg;
                // The streamed variant keeps as many leading rows as its LDS
                // holds (or a.lds_rows when set) and streams the rest.
                const size_t base = pipe_lds_bytes(pi.m, rmax, P4, ldsw);
                int rl = ldsw ? rmax : 0;
                if (!ldsw && base < (size_t)max_lds) {
                    const int64_t fit = ((int64_t)max_lds - (int64_t)base) / (P4 * 16);
                    rl = (int)(fit < rmax ? fit : rmax);
                    if (a.lds_rows >= 0) rl = a.lds_rows < rl ? a.lds_rows : rl;
                }
                if (rmax <= 64 && base <= (size_t)max_lds) {
                    // Calibrated on MI355X (LDS and streamed kernels, block
                    // lengths 2 to 8, 2 to 256 workgroups).  Sweepers: one
                    // pass over the rows per block, a row costing
                    // KS (0.027 M + 0.04) + 0.012 M + 0.067 us, plus
                    // 0.5 + 0.15 M us of hand-over per block and 0.05 us per
                    // streamed row, and at least the read and write of the
                    // streamed rows at the workgroup's share of 8 TB/s.
                    // Controller: one exchange per step plus 0.03 M us
                    // (longer blocks' larger unrolled code) and 0.36 us per
                    // block.  A step takes the slower of the two.
                    const double row_us = ks_need * (0.027 * pi.m + 0.0395) + 0.012 * pi.m + 0.0665;
                    const double blk_us =
                        rmax * row_us + (rmax - rl) * 0.05 + 0.5 + 0.15 * pi.m;
                    const double mem_us = (rmax - rl) * P4 * 32.0 / (8e6 / gg);
                    const double sweep = (blk_us > mem_us ? blk_us : mem_us) / pi.m;
                    const double ctl = pipe_exchange_us(gg) + 0.03 * pi.m + 0.36 / pi.m;
                    const double t = sweep > ctl ? sweep : ctl;
                    if (t < best) {
                        best = t;
                        plan->grid = gg;
                        plan->variant = ldsw ? 3 : 2;
                        plan->block_m = pi.m;
                        plan->kslots = pi.ks;
                        plan->lds_rows = ldsw ? 0 : rl;
                        plan->block = 256;
                    }
                }
                if (a.grid > 0 || g >= max_grid) break;
            }
        }
    }
    // Four sweepers for the streamed rows: the same pass split over four
    // waves instead of three, on every SIMD, the controller beside the
    // first sweeper.  Cost as above with the four-sweeper slice count and
    // the first sweeper's rows 12 % slower (the controller's issue slots
    // on its SIMD).  Only where rows are streamed (unless four sweepers are
    // asked for): with every row in LDS the LDS-resident kernel, whose
    // exchanges keep four polls in flight, measured faster (20 x 20 map,
    // d = 2000, 64 workgroups: 1.29 against 1.74 us per step).
    for (const Wide &wi : kWide) {
        const int ks4 = (nsl + 3) / 4;
        if (wi.ks != ks4 || a.variant == 1 || a.sweepers == 3 ||
            (a.block_m > 0 && wi.m != a.block_m))
            continue;
        for (int g = 1;; g = (g * 2 > max_grid && g < max_grid) ? max_grid : g * 2) {
            const int gg = a.grid > 0 ? (a.grid < a.N ? a.grid : a.N) : g;
            const int rmax = (a.N + gg - 1) / gg;
            const size_t base = pipe_lds_bytes(wi.m, rmax, P4, false, false, 4);
            int rl = 0;
            if (base < (size_t)max_lds) {
                const int64_t fit = ((int64_t)max_lds - (int64_t)base) / (P4 * 16);
                rl = (int)(fit < rmax ? fit : rmax);
                if (a.lds_rows >= 0) rl = a.lds_rows < rl ? a.lds_rows : rl;
            }
            if (rmax <= 64 && base <= (size_t)max_lds && (rl < rmax || a.sweepers == 4)) {
                const double row_us = 1.12 * (ks4 * (0.027 * wi.m + 0.0395) + 0.012 * wi.m + 0.0665);
                const double blk_us = rmax * row_us + (rmax - rl) * 0.05 + 0.5 + 0.15 * wi.m;
                const double mem_us = (rmax - rl) * P4 * 32.0 / (8e6 / gg);
                const double sweep = (blk_us > mem_us ? blk_us : mem_us) / wi.m;
                const double ctl = pipe_exchange_us(gg) + 0.03 * wi.m + 0.36 / wi.m;
                const double t = sweep > ctl ? sweep : ctl;
                if (t < best) {
                    best = t;
                    plan->grid = gg;
                    plan->variant = 2;
                    plan->block_m = wi.m;
                    plan->kslots = wi.ks;
                    plan->lds_rows = rl;
                    plan->block = 320;
                }
            }
            if (a.grid > 0 || g >= max_grid) break;
        }
    }
    // Rows too long for any instance above (their sample slices would not
    // fit in registers): the column-walk sweep, rows streamed with the first
    // few kept in LDS, when the workgroups own few enough rows.  Cost:
    // about 0.0085 (3 M + 3) us per row and slice of 64 float4 per sweeper
    // (3 M + 2 VALU operations per element and block, and the loop's
    // overhead), 0.07 us per row for the lane sums, 0.5 us of hand-over per
    // block, and at least the streamed rows' read and write at the
    // workgroup's share of 6.8 TB/s (the in-place stream rate of a
    // MALL-resident footprint); the controller as above.
    const bool no_rows_instance = best >= 1e300;
    for (const ColsInstance &ci : kCols) {
        if (!no_rows_instance || a.variant == 1) break;
        if (a.block_m > 0 && ci.m != a.block_m) continue;
        for (int g = 1;; g = (g * 2 > max_grid && g < max_grid) ? max_grid : g * 2) {
            const int gg = a.grid > 0 ? (a.grid < a.N ? a.grid : a.N) : g;
            const int rmax = (a.N + gg - 1) / gg;
            const size_t base = pipe_lds_bytes(ci.m, rmax, P4, false, true);
            if (rmax <= ci.rmax && base <= (size_t)max_lds) {
                int64_t fit = ((int64_t)max_lds - (int64_t)base) / (P4 * 16);
                if (fit > kColsLdsRows) fit = kColsLdsRows;
                int rl = (int)(fit < rmax ? fit : rmax);
                if (a.lds_rows >= 0) rl = a.lds_rows < rl ? a.lds_rows : rl;
                const double blk_us = rmax * (ks_need * 0.0085 * (3 * ci.m + 3) + 0.07) + 0.5;
                const double mem_us = (rmax - rl) * P4 * 32.0 / (6.8e6 / gg);
                const double sweep = (blk_us > mem_us ? blk_us : mem_us) / ci.m;
                const double ctl = pipe_exchange_us(gg) + 0.03 * ci.m + 0.36 / ci.m;
                const double t = sweep > ctl ? sweep : ctl;
                if (t < best) {
                    best = t;
                    plan->grid = gg;
                    plan->variant = 4;
                    plan->block_m = ci.m;
                    plan->kslots = 0;
                    plan->lds_rows = rl;
                    plan->cols_rmax = ci.rmax;
                    plan->block = 256;
                }
            }
            if (a.grid > 0 || g >= max_grid) break;
        }
    }
    if (best < 1e300 && plan->cols_rmax > 0) {
        plan->lds_bytes = pipe_lds_bytes(plan->block_m, (a.N + plan->grid - 1) / plan->grid, P4,
                                          false, true) +
                          (size_t)plan->lds_rows * P4 * 16;
        if (plan->lds_bytes < 84 * 1024) plan->lds_bytes = 84 * 1024;
        plan->block = 256;
        plan->slot_spread = plan->grid <= 64 ? 16 : 4;
        PipeKernel fn = pipe_cols_kernel(plan->block_m, plan->cols_rmax);
        int per_cu = 0;
        if (!fn ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &per_cu, reinterpret_cast<const void *>(fn), 256, plan->lds_bytes) != hipSuccess ||
            per_cu < 1 || plan->grid > per_cu * num_cus || plan->grid > kMaxTrainGrid)
            return 1e300;
        return best;
    }
    if (best < 1e300) {
        const int ns = plan->block / 64 - 1;
        plan->lds_bytes = pipe_lds_bytes(plan->block_m, (a.N + plan->grid - 1) / plan->grid, P4,
                                          plan->variant == 3, false, ns) +
                          (size_t)plan->lds_rows * P4 * 16;
        if (plan->lds_bytes < 84 * 1024) plan->lds_bytes = 84 * 1024;
        // Measured on MI355X: the LDS-resident kernels' multi-poll exchanges
        // are fastest with packed slots, the streamed kernels' one-poll
        // exchanges with one slot per 128-byte line up to 64 workgroups and
        // 32-byte spacing beyond.
        plan->slot_spread = plan->variant == 3 ? 1 : (plan->grid <= 64 ? 16 : 4);
        PipeKernel fn = nullptr;
        if (plan->variant == 3) {
            const PipeInstance *pi = pipe_for(plan->block_m, plan->kslots);
            fn = pi ? pi->lds : nullptr;
        } else {
            fn = pipe_stream_kernel(plan->block_m, plan->kslots, ns);
        }
        int per_cu = 0;
        if (!fn ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &per_cu, reinterpret_cast<const void *>(fn), plan->block, plan->lds_bytes) !=
                hipSuccess ||
            per_cu < 1 || plan->grid > per_cu * num_cus || plan->grid > kMaxTrainGrid)
            return 1e300;
    }
    return best;
}

int64_t pipe_block_dots_floats(int m, int64_t nsteps) {
    const int64_t nb = (nsteps + m - 1) / m;
    return nb * (m * (m + 1) + m * m);
}

hipError_t launch_train_pipe(const TrainArgs &a, const TrainPlan &plan, hipStream_t s) {
    const int64_t P4 = a.ld / 4;
    if (plan.cols_rmax > 0) {
        // long rows: the column-walk sweep (its prepass is the same)
        PipeKernel fn = pipe_cols_kernel(plan.block_m, plan.cols_rmax);
        DotsKernel dots = block_dots_for(plan.block_m);
        if (!fn || !dots || !a.block_dots || P4 % 64 != 0 || a.xld != a.ld ||
            (a.N + plan.grid - 1) / plan.grid > plan.cols_rmax || plan.variant != 4 ||
            plan.lds_rows > kColsLdsRows)
            return hipErrorInvalidValue;
        TrainArgs args = a;
        args.grid = plan.grid;
        args.slot_spread = plan.slot_spread;
        args.lds_rows = plan.lds_rows;
        const int64_t nb = (a.nsteps + plan.block_m - 1) / plan.block_m;
        dots<<<dim3((unsigned)nb), dim3(256), 0, s>>>(args, args.block_dots, nb);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        void *params[] = {&args};
        return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(fn),
                                          dim3(plan.grid - plan.absent), dim3(256), params,
                                          (unsigned)plan.lds_bytes, s);
    }
    const int ns = plan.block / 64 - 1;
    if (ns != 3 && ns != 4) return hipErrorInvalidValue;
    DotsKernel dots = block_dots_for(plan.block_m);
    const PipeInstance *pi = pipe_for(plan.block_m, plan.kslots);
    PipeKernel fn = plan.variant == 3 ? (pi && ns == 3 ? pi->lds : nullptr)
                                      : pipe_stream_kernel(plan.block_m, plan.kslots, ns);
    if (!fn || !dots || !a.block_dots) return hipErrorInvalidValue;
    if (P4 % 64 != 0 || (P4 / 64 + ns - 1) / ns != plan.kslots ||
        (a.N + plan.grid - 1) / plan.grid > 64)
        return hipErrorInvalidValue;
    TrainArgs args = a;
    args.grid = plan.grid;
    args.slot_spread = plan.slot_spread;
    args.lds_rows = plan.variant == 3 ? 0 : plan.lds_rows;
    const int64_t nb = (a.nsteps + plan.block_m - 1) / plan.block_m;
    dots<<<dim3((unsigned)nb), dim3(256), 0, s>>>(args, args.block_dots, nb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    void *params[] = {&args};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(fn),
                                      dim3(plan.grid - plan.absent), dim3(plan.block), params,
                                      (unsigned)plan.lds_bytes, s);
}

}  // namespace som
