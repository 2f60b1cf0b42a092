// Device helpers shared by the training kernels: wave reductions, per-step
// input windows, sample loads, the grid exchange and the neighbourhood
// factor.  Included by the kernel translation units only.
#pragma once

#include "som_internal.h"

#include <math.h>
#include <type_traits>

namespace som {
namespace dev {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int32_t kStatusTimeout = 5;  // SOM_E_TIMEOUT

// Prototype rows live either in LDS or in global memory.  Pointers typed
// with the address space make the compiler use LDS (ds_*) or global
// instructions instead of generic (flat) ones, which count against both
// memory counters and so make every wait for a row also wait for any
// outstanding sample load.
template <bool LDS>
struct RowSpace {
    typedef __attribute__((address_space(1))) f4 T;
};
template <>
struct RowSpace<true> {
    typedef __attribute__((address_space(3))) f4 T;
};
template <bool LDS>
using row_t = typename RowSpace<LDS>::T;
template <bool LDS>
__device__ inline row_t<LDS> *rows_as(f4 *p) {
    return (row_t<LDS> *)p;
}

// Sums over the 64 lanes of a wave, for U values at once, returned to every
// lane.  Within each row of 16 lanes a butterfly of DPP moves (quad swaps,
// half-row and row mirrors) leaves the row's sum in all of its lanes,
// bit-identical because every pairwise add is commutative; the four row sums
// are then read out and added in a fixed order.  The U chains run in
// lockstep so their DPP hazards overlap.
template <int CTRL>
__device__ inline int dpp_move(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xf, 0xf, false);
}
template <int CTRL>
__device__ inline float dpp_pair(float v) {
    return v + __int_as_float(dpp_move<CTRL>(__float_as_int(v)));
}
__device__ inline float lane_f(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
template <int U>
__device__ inline void wave_sums(float (&v)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_pair<0xB1>(v[u]);   // quad_perm [1,0,3,2]
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_pair<0x4E>(v[u]);   // quad_perm [2,3,0,1]
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_pair<0x141>(v[u]);  // row_half_mirror
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_pair<0x140>(v[u]);  // row_mirror
#pragma unroll
    for (int u = 0; u < U; ++u)
        v[u] = (lane_f(v[u], 0) + lane_f(v[u], 16)) + (lane_f(v[u], 32) + lane_f(v[u], 48));
}

// As wave_sums, but the sums are complete only in lane 63: after the row
// butterflies, row_bcast:15 adds each row's last lane into rows 1 and 3 and
// row_bcast:31 adds lane 31 into rows 2 and 3 (six DPP adds per value
// instead of four adds, four lane reads and three adds).
template <int CTRL, int ROWS>
__device__ inline float dpp_add_rows(float v) {
    return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROWS, 0xf,
                                                          false));
}
template <int U>
__device__ inline void wave_sums_last(float (&v)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_pair<0xB1>(v[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_pair<0x4E>(v[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_pair<0x141>(v[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_pair<0x140>(v[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_add_rows<0x142, 0xa>(v[u]);  // row_bcast:15
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_add_rows<0x143, 0xc>(v[u]);  // row_bcast:31
}

// Sums over the 64 lanes of U values, left in (U + 3) / 4 registers: the
// sum of v[k] ends up in every lane of row sum_row(k) (lanes 16 row ..
// 16 row + 15) of t[k / 4].  Lanes l and l + 32 are added first, pairing
// the values two by two through a permlane32 swap (one swap and one add per
// pair), then rows 0/1 and 2/3 the same way through a permlane16 swap, and
// last the 16 lanes of each row by the DPP butterfly: about 1.5 U + 4 U / 4
// instructions instead of the 6 U of a butterfly per value.
constexpr int sum_row(int k) { return (k & 1) * 2 + ((k >> 1) & 1); }

__device__ inline void swap_halves(float &a, float &b) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b),
                                                     false, false);
    a = __uint_as_float(r[0]);  // lanes 0-31: a's, 32-63: b's lanes 0-31
    b = __uint_as_float(r[1]);  // lanes 0-31: a's lanes 32-63, 32-63: b's
}
__device__ inline void swap_rows(float &a, float &b) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b),
                                                     false, false);
    a = __uint_as_float(r[0]);  // rows: a0 b0 a2 b2
    b = __uint_as_float(r[1]);  // rows: a1 b1 a3 b3
}
template <int U>
__device__ inline void wave_sums_rows(const float (&v)[U], float (&t)[(U + 3) / 4]) {
    constexpr int S1 = (U + 1) / 2, S2 = (S1 + 1) / 2;
    static_assert(S2 == (U + 3) / 4, "two halvings");
    float h[S1];
#pragma unroll
    for (int i = 0; i < S1; ++i) {
        float a = v[2 * i], b = 2 * i + 1 < U ? v[2 * i + 1] : 0.f;
        swap_halves(a, b);
        h[i] = a + b;  // lanes 0-31: v[2i], 32-63: v[2i+1], each over lanes l, l + 32
    }
#pragma unroll
    for (int j = 0; j < S2; ++j) {
        float a = h[2 * j], b = 2 * j + 1 < S1 ? h[2 * j + 1] : 0.f;
        swap_rows(a, b);
        t[j] = a + b;  // rows: v[4j], v[4j+2], v[4j+1], v[4j+3] over 4 lanes each
    }
#pragma unroll
    for (int j = 0; j < S2; ++j) t[j] = dpp_pair<0xB1>(t[j]);   // quad_perm [1,0,3,2]
#pragma unroll
    for (int j = 0; j < S2; ++j) t[j] = dpp_pair<0x4E>(t[j]);   // quad_perm [2,3,0,1]
#pragma unroll
    for (int j = 0; j < S2; ++j) t[j] = dpp_pair<0x141>(t[j]);  // row_half_mirror
#pragma unroll
    for (int j = 0; j < S2; ++j) t[j] = dpp_pair<0x140>(t[j]);  // row_mirror
}

__device__ inline unsigned long long u64_min(unsigned long long a, unsigned long long b) {
    return a < b ? a : b;
}

// Minimum over the 64 lanes of a wave (same DPP pattern), to every lane.
__device__ inline unsigned wave_min_u32(unsigned v) {
    v = min(v, (unsigned)dpp_move<0xB1>((int)v));
    v = min(v, (unsigned)dpp_move<0x4E>((int)v));
    v = min(v, (unsigned)dpp_move<0x141>((int)v));
    v = min(v, (unsigned)dpp_move<0x140>((int)v));
    const unsigned a = (unsigned)__builtin_amdgcn_readlane((int)v, 0);
    const unsigned b = (unsigned)__builtin_amdgcn_readlane((int)v, 16);
    const unsigned c = (unsigned)__builtin_amdgcn_readlane((int)v, 32);
    const unsigned d = (unsigned)__builtin_amdgcn_readlane((int)v, 48);
    return min(min(a, b), min(c, d));
}

// Minimum of a 64-bit key over the wave: the high words first, then the low
// words among the lanes that hold the minimal high word.  When the low words
// increase with the lane (lanes_ordered), or only one lane holds the minimal
// high word, that is the low word of the first such lane.
__device__ inline unsigned long long wave_min_key(unsigned long long v, bool lanes_ordered) {
    const unsigned hi = (unsigned)(v >> 32), lo = (unsigned)v;
    const unsigned mh = wave_min_u32(hi);
    const unsigned long long hit = __ballot(hi == mh);
    unsigned ml;
    if (lanes_ordered || __builtin_popcountll(hit) == 1)
        ml = (unsigned)__builtin_amdgcn_readlane((int)lo, __builtin_ctzll(hit));
    else
        ml = wave_min_u32(hi == mh ? lo : 0xffffffffu);
    return ((unsigned long long)mh << 32) | ml;
}

// Distance bits that compare as unsigned integers in the order of the
// distances: NaN counts as +inf, -0 as +0, and a negative value (the
// rounding of a near-zero distance in Gram form) below every positive one.
__device__ inline unsigned dist_order_bits(float D) {
    const unsigned b = __float_as_uint(fminf(D, INFINITY) + 0.f);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Key (distance bits << 32 | unit) of the smallest of the lanes' distance
// bits, ties to the lowest lane; lane l stands for unit u0 + l.  Idle lanes
// pass 0xffffffff, which no distance maps to; lane 0 must not be idle.
__device__ inline unsigned long long wave_argmin_key(unsigned bits, int u0) {
    const unsigned m = wave_min_u32(bits);
    const unsigned long long hit = __ballot(bits == m);
    return ((unsigned long long)m << 32) | (unsigned)(u0 + __builtin_ctzll(hit));
}

typedef const __attribute__((address_space(1))) float gfloat;
typedef const __attribute__((address_space(1))) f4 gf4;

// Loads that may fall past the end of a row are made at a clamped column
// and then replaced by zero with a select: a load under a branch joins the
// zero of the other path in a copy that waits for the load, which
// serialises a burst of loads into one memory round trip each.
__device__ inline f4 load_f4_or_zero(gf4 *row, int q, int n4) {
    const f4 v = row[q < n4 ? q : n4 - 1];
    const f4 zero = {0.f, 0.f, 0.f, 0.f};
    return q < n4 ? v : zero;
}
// float4 column q of sample row i (zero past the row's xld / 4 columns).
__device__ inline f4 sample_f4(const TrainArgs &a, int64_t i, int q) {
    return load_f4_or_zero((gf4 *)(a.X + i * a.xld), q, (int)(a.xld >> 2));
}

// Sample row i into the lane's slots; columns past d (row padding) are 0.
template <int K, int L>
__device__ inline void load_sample(f4 (&x)[K], const TrainArgs &a, int64_t i) {
    const int li = threadIdx.x % L;
#pragma unroll
    for (int k = 0; k < K; ++k) x[k] = sample_f4(a, i, li + L * k);
}

// Per-step inputs (sample index, schedule entry) are fetched 64 steps at a
// time: lane l of a window holds the entry of step base + l, loaded with one
// vector load, and a step's entry is read out with readlane.  Vector loads
// keep these fetches off the scalar-memory counter that LDS operations
// share, so waiting for LDS never waits for them.  The next window is
// loaded while the current one is in use.
__device__ inline int fetch_entry(const TrainArgs &a, int64_t s, int) {
    int i = s < a.nsteps ? a.order[s] : 0;
    return (i >= 0 && (int64_t)i < a.n) ? i : 0;  // range-checked before launch
}
__device__ inline float2 fetch_entry(const TrainArgs &a, int64_t s, float2) {
    return s < a.nsteps ? a.sched[s] : make_float2(0.f, 0.f);
}

template <typename T>
struct StepWindow {
    int64_t base;
    T cur, next;

    __device__ void init(const TrainArgs &a, int64_t b) {
        base = b;
        cur = fetch_entry(a, b + (threadIdx.x & 63), T());
        next = fetch_entry(a, b + 64 + (threadIdx.x & 63), T());
    }
    // Entry of step s, for non-decreasing s >= base.
    __device__ T get(const TrainArgs &a, int64_t s) {
        if (s >= base + 64) {
            base += 64;
            cur = next;
            next = fetch_entry(a, base + 64 + (threadIdx.x & 63), T());
        }
        return lane_value((int)(s - base));
    }
    __device__ T lane_value(int l) const;
};

template <>
__device__ inline int StepWindow<int>::lane_value(int l) const {
    return __builtin_amdgcn_readlane(cur, l);
}
template <>
__device__ inline float2 StepWindow<float2>::lane_value(int l) const {
    return make_float2(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(cur.x), l)),
                       __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cur.y), l)));
}


// Packed index of the Gram entry (i, j), i <= j.
__device__ constexpr int tri(int i, int j) { return j * (j + 1) / 2 + i; }
__device__ constexpr int tri_any(int i, int j) { return i <= j ? tri(i, j) : tri(j, i); }

__device__ inline unsigned long long row_key(float D, int u) {
    return ((unsigned long long)dist_order_bits(D) << 32) | (unsigned)u;
}

// Lattice row and column of unit c < 2^24: the fp32 quotient c * (1 / cols)
// is within one of c / cols (both roundings are exact for cols <= 2 and
// the error stays below 2^24 / cols * 2^-23 < 1 otherwise), so one
// correction step makes it exact.
__device__ inline void unit_rc(int c, int cols, float inv_cols, int &r, int &col) {
    int q = (int)((float)c * inv_cols);
    int rem = c - q * cols;
    if (rem < 0) {
        --q;
        rem += cols;
    } else if (rem >= cols) {
        ++q;
        rem -= cols;
    }
    r = q;
    col = rem;
}

struct Bcast {
    int abort;
    int pad[3];
};

// One wave per workgroup: publish this workgroup's best key to grid
// exchange number e (the two halves of exchange() below, for callers that
// work between them).
__device__ inline void exchange_publish(const TrainArgs &a, int64_t e, unsigned long long best) {
    const int lane = threadIdx.x & 63, G = a.grid;
    if (G == 1) return;
    const unsigned tag = 0x80u | (unsigned)((e >> 1) & 0x7f);
    const int sp = a.slot_spread;
    const int64_t par = (e & 1) * (int64_t)G * sp;
    if (lane < kSlotReplicas) {
        const unsigned long long v = (best & 0xffffffff00000000ull) |
                                     ((unsigned long long)tag << kUnitBits) |
                                     (best & (unsigned long long)kMaxUnits);
        __hip_atomic_store(a.slots + lane * kSlotReplicaStride + par + (int64_t)blockIdx.x * sp,
                           v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Poll the slots base + lane + 64 k (k < K) of one exchange until every
// lane has the key of each of its slots that exists, folding the keys into
// m.  P polls per lane (4 or 8) are in flight, position q reading slot
// q % K, so all of a group's slots are read in the same memory round trip
// and each check waits only for the oldest poll, whose replacement goes out
// right after it.  Control flow stays wave-uniform (the wave leaves once no
// lane misses a key): per-lane exits would make the compiler copy the
// in-flight values, and every copy waits for its load.  The positions are
// unrolled by hand so that each exit is a plain break, and the translation
// units that use this are built with uniform regions left unstructured;
// exits merged into the loop latch would make the compiler wait for every
// poll at the loop head.  Returns 0, or 1 if the map's status word turned
// non-zero, or 2 on timeout.
template <int q>
using Pos = std::integral_constant<int, q>;

// The registers an exchange polls into, kept by the caller from one
// exchange to the next.  An exchange returns with polls still in flight;
// were their registers free, the compiler would reuse them at once and wait
// for those polls first (a memory round trip for the newest).  Held by the
// caller, they stay untouched until the next exchange, which lets them land
// (a load into a register whose previous load is still in flight needs no
// wait) and marks them used only where they have landed anyway.
template <int P>
struct PollRegs {
    unsigned long long v[P];
};
template <>
struct PollRegs<1> {};

// s_waitcnt immediate for vmcnt(0) with the other counters left alone
// (expcnt 7, lgkmcnt 15): wait for every vector memory operation in flight.
constexpr unsigned kWaitVmemAll = 0x0F70;

template <int K, int P, typename Work>
__device__ __forceinline__ int poll_slots(const TrainArgs &a, const unsigned long long *slots,
                                          int base, unsigned tag, unsigned long long &m,
                                          Work &&work, PollRegs<P> &pr) {
    static_assert(P == 4 || P == 8, "four or eight polls in flight");
    const int lane = threadIdx.x & 63, G = a.grid, sp = a.slot_spread;
    const unsigned long long *adr[K];
    unsigned need = 0;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int i = base + lane + 64 * k;
        const bool mine = i < G;
        adr[k] = slots + (int64_t)(mine ? i : base) * sp;
        need |= mine ? 1u << k : 0u;
    }
    unsigned long long(&v)[P] = pr.v;  // the caller's registers
#pragma unroll
    for (int q = 0; q < P; ++q)
        v[q] = __hip_atomic_load(adr[q % K], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    work();  // the caller's work, while the first polls are in flight
    // Check position q and put its next poll in flight (before the exit
    // test: a poll skipped on the way out would leave the loop head unsure
    // which load is the oldest); true once no lane misses a key.
    const auto step = [&](auto pos) {
        constexpr int q = decltype(pos)::value;
        constexpr unsigned bit = 1u << (q % K);
        const bool ok = (need & bit) != 0 && ((unsigned)(v[q] >> kUnitBits) & 0xffu) == tag;
        m = ok ? u64_min(m, v[q]) : m;
        need &= ok ? ~bit : ~0u;
        const bool done = __ballot(need != 0) == 0;
        v[q] = __hip_atomic_load(adr[q % K], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return done;
    };
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    int r = 0;
    for (unsigned spins = 1;; ++spins) {
        if ((spins & 15u) == 0) {
            const int32_t st =
                __hip_atomic_load(&a.state->status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (__ballot(st != 0) != 0) {
                r = 1;
                break;
            }
            if (__builtin_amdgcn_s_memrealtime() - t0 > a.timeout_ticks) {
                r = 2;
                break;
            }
        }
        if (step(Pos<0>{})) break;
        if (step(Pos<1>{})) break;
        if (step(Pos<2>{})) break;
        if (step(Pos<3>{})) break;
        if constexpr (P == 8) {
            if (step(Pos<4>{})) break;
            if (step(Pos<5>{})) break;
            if (step(Pos<6>{})) break;
            if (step(Pos<7>{})) break;
        }
    }
    return r;
}

// Wait for every workgroup's key of exchange e and return the winning unit
// (the same in all lanes), or -1 if the wait was given up.  `best` is this
// workgroup's own key (the answer when the grid is one workgroup).  `work`
// (independent of the result) runs once, while the wait is under way.  P polls
// per lane are kept in flight: 4 or 8, or 1 (each lane waits for its slots
// one after the other: the fewest registers and the least polling traffic).
template <int P, typename Work>
__device__ __forceinline__ int exchange_wait(const TrainArgs &a, int64_t e,
                                             unsigned long long best, Work &&work,
                                             PollRegs<P> &pr) {
    const int lane = threadIdx.x & 63, G = a.grid;
    if (G == 1) {
        work();
        return (int)(best & (unsigned long long)kMaxUnits);
    }
    const unsigned tag = 0x80u | (unsigned)((e >> 1) & 0x7f);
    const int64_t par = (e & 1) * (int64_t)G * a.slot_spread;
    const unsigned long long *slots =
        a.slots + (blockIdx.x % kSlotReplicas) * kSlotReplicaStride + par;
    unsigned long long m = ~0ull;
    int abort = 0;
    const auto none = [] {};
    if constexpr (P == 1) {
        // One poll per lane at a time, each lane waiting for its slots one
        // after the other: the fewest registers.
        work();
        const int sp = a.slot_spread;
        for (int i = lane; i < G && abort == 0; i += 64) {
            const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
            for (unsigned spins = 1;; ++spins) {
                const unsigned long long v = __hip_atomic_load(
                    slots + (int64_t)i * sp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (((unsigned)(v >> kUnitBits) & 0xffu) == tag) {
                    m = u64_min(m, v);
                    break;
                }
                if ((spins & 63u) == 0) {
                    if (__hip_atomic_load(&a.state->status, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT) != 0) {
                        abort = 1;
                        break;
                    }
                    if (__builtin_amdgcn_s_memrealtime() - t0 > a.timeout_ticks) {
                        abort = 2;
                        break;
                    }
                }
            }
        }
    } else if (G <= 256) {
        // One group, and no loop around it (a loop head would make the
        // compiler wait for every memory operation in flight).  Polling
        // starts at once on small grids; beyond 16 workgroups it starts
        // after this workgroup's key stores have completed, which measures
        // faster there (the early polls only add traffic on the slot lines
        // while the other workgroups' stores are still landing).
        // The caller's work runs while the key stores complete, or on small
        // grids while the first polls are in flight.
        if (G > 16) {
            work();
            __builtin_amdgcn_s_waitcnt(kWaitVmemAll);
            // the previous exchange's polls have landed with everything else
#pragma unroll
            for (int q = 0; q < P; ++q) asm volatile("" ::"v"(pr.v[q]));
            abort = G <= 64    ? poll_slots<1, P>(a, slots, 0, tag, m, none, pr)
                    : G <= 128 ? poll_slots<2, P>(a, slots, 0, tag, m, none, pr)
                               : poll_slots<4, P>(a, slots, 0, tag, m, none, pr);
        } else {
            // Small grids poll at once: a use of the previous exchange's
            // poll registers waits only for those of its polls still in
            // flight, which have had a step's work to land.
#pragma unroll
            for (int q = 0; q < P; ++q) asm volatile("" ::"v"(pr.v[q]));
            abort = poll_slots<1, P>(a, slots, 0, tag, m, work, pr);
        }
    } else {
        // groups of 256 (slots past the grid count as received)
        work();
#pragma unroll
        for (int q = 0; q < P; ++q) asm volatile("" ::"v"(pr.v[q]));
        for (int base = 0; base < G && abort == 0; base += 256)
            abort = poll_slots<4, P>(a, slots, base, tag, m, none, pr);
    }
    // The timeout is recorded after the polls: a store among them would mix
    // stores into the loads in flight, and the compiler then waits for every
    // poll at each check.
    if (abort == 2)
        __hip_atomic_store(&a.state->status, kStatusTimeout, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    // With at most 64 workgroups lane i holds workgroup i's key, and
    // workgroups own increasing unit ranges.
    m = wave_min_key(m, G <= 64);
    if (__ballot(abort) != 0) return -1;
    return (int)(m & (unsigned long long)kMaxUnits);
}

// Publish this workgroup's best key to grid exchange number e and return
// the winning unit over every workgroup's slot, or -1 if the wait was given
// up.  Each workgroup writes its key into every XCD's copy of the slot
// array and polls the copy of its own XCD; slots alternate by the parity
// of e and carry a tag of e, so a slot is never read for the wrong step.
template <int P>
__device__ inline int exchange(const TrainArgs &a, int64_t e, unsigned long long best,
                               PollRegs<P> &pr) {
    exchange_publish(a, e, best);
    return exchange_wait<P>(a, e, best, [] {}, pr);
}

// Neighbourhood factor of owned row r given BMU c: lr * 2^(-g * c2) with g
// the squared lattice distance.  pos[r] holds (row, column, row parity) of
// unit r0 + r.  RECT: g = dr^2 + dc^2.  HEX: odd rows shifted by 1/2 and rows
// sqrt(3)/2 apart, so g = 3/4 dr^2 + (dc + (parity difference) / 2)^2, exact
// in fp32 for the map sizes the library accepts.
__device__ inline float neighbour_h(const TrainArgs &a, float4 p, float cr, float cc,
                                    float cpar, float lr, float c2) {
    const float dr = p.x - cr;
    float dx = p.y - cc, g;
    if (a.topology == 1) {
        dx += 0.5f * (p.z - cpar);
        g = 0.75f * dr * dr + dx * dx;
    } else {
        g = dr * dr + dx * dx;
    }
    // v_exp_f32 directly: results below the normal range flush to zero
    // (a neighbourhood factor under 2^-126 moves nothing in fp32 anyway).
    return lr * __builtin_amdgcn_exp2f(-g * c2);
}

// One wave per workgroup runs the mb steps s0 .. s0 + mb - 1 of a block from
// the Gram matrices E of the workgroup's rows (lane r holds row r < R, with
// lattice position p), leaving the block's coefficients in (beta, gam):
// after the block a prototype is w_end = beta w_start + sum_j gam_j x_j.
// Step k's distance D_k = E_kk - 2 sum_j gam_j E_jk + sum_ij gam_i gam_j E_ij
// is carried from step to step through lin_l = sum_j gam_j E_jl and
// quad = sum_ij gam_i gam_j E_ij: a step with factor h scales every gam by
// (1 - h) and sets gam_k = h, so
//   quad <- (1 - h)^2 quad + 2 h (1 - h) lin_k + h^2 E_kk,
//   lin_l <- (1 - h) lin_l + h E_kl.
// Returns false if an exchange was given up.  P: polls in flight per lane
// in each exchange, into the caller's registers pr.
template <int M, int P>
__device__ inline bool block_steps(const TrainArgs &a, int64_t s0, int mb, int r0, int R,
                                   const float (&E)[M * (M + 1) / 2], float4 p, float inv_cols,
                                   StepWindow<float2> &sw, float &beta, float (&gam)[M],
                                   PollRegs<P> &pr) {
    const int lane = threadIdx.x & 63;
    float lin[M], quad = 0.f;
    beta = 1.f;
#pragma unroll
    for (int j = 0; j < M; ++j) {
        gam[j] = 0.f;
        lin[j] = 0.f;
    }
    if (mb <= 0) return true;
    const auto key_of = [&](float D) {
        return wave_argmin_key(lane < R ? dist_order_bits(D) : 0xffffffffu, r0);
    };
    // Each step publishes the next step's key as soon as its distance is
    // known (it needs only quad and lin_{k+1}); the rest of its bookkeeping
    // runs inside the next exchange's wait, off the path from one exchange
    // to the next.  Step 0's distance is E_00 (no step taken yet).
    const auto book = [&](int k, float h, float om) {
#pragma unroll
        for (int l = k + 2; l < M; ++l) lin[l] = fmaf(h, E[tri(k, l)], om * lin[l]);
        beta *= om;
#pragma unroll
        for (int j = 0; j < k; ++j) gam[j] *= om;
        gam[k] = h;
    };
    float2 sc = sw.get(a, s0);
    unsigned long long best = key_of(E[tri(0, 0)]);
    exchange_publish(a, s0, best);
    bool ok = true;
    float h_prev = 0.f, om_prev = 1.f;
#pragma unroll
    for (int k = 0; k < M; ++k) {
        if (k >= mb || !ok) continue;
        const int64_t s = s0 + k;
        const int c = exchange_wait<P>(
            a, s, best,
            [&] {
                if (k > 0) book(k - 1, h_prev, om_prev);
            },
            pr);
        if (c < 0) {
            ok = false;
            continue;
        }
        int cr, cc;
        unit_rc(c, a.cols, inv_cols, cr, cc);
        const float h = neighbour_h(a, p, (float)cr, (float)cc, (float)(cr & 1), sc.x, sc.y);
        const float om = 1.f - h;
        quad = fmaf(om * om, quad, h * fmaf(2.f * om, lin[k], h * E[tri(k, k)]));
        if (k + 1 < M) lin[k + 1] = fmaf(h, E[tri(k, k + 1)], om * lin[k + 1]);
        if (k + 1 < mb) {
            sc = sw.get(a, s + 1);
            best = key_of(fmaf(-2.f, lin[k + 1], E[tri(k + 1, k + 1)]) + quad);
            exchange_publish(a, s + 1, best);
            h_prev = h;
            om_prev = om;
        } else {
            book(k, h, om);  // the block's last step: no wait follows
        }
        if (blockIdx.x == 0 && lane == 0 && a.bmu_trace) a.bmu_trace[s] = c;
    }
    return ok;
}

}  // namespace dev
}  // namespace som
