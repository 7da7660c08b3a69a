// gfx950 kernels of the collective hot path.
//
// * reduce_step_kernel -- one ring reduction step for every virtual rank at
//   once: out[i] = in0[i] + in1[i], where in0 is the partial received from
//   the previous rank (or, on the first step, that rank's own element) and
//   in1 is this rank's element.  bf16 partials are carried in fp32.
// * fold_kernel        -- the direct variant: folds all R inputs of a chunk
//   in the ring order in one pass (same result bit for bit, fewer bytes).
// * copy_kernel        -- a CU copy of many independent (src, dst, bytes)
//   segments; the comparator for the SDMA copy path.
//
// All three are HBM-bound streams (about one add per 8-12 bytes), so they
// use 16-byte vector loads and stores, a grid-stride loop over each segment
// with several independent vectors in flight per thread, and no LDS and no
// MFMA: the limit is memory bandwidth, not arithmetic.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "hoccl_internal.h"

namespace hoccl {
namespace {

// ---- element types ----------------------------------------------------------
// S is the storage type in memory, A the accumulator type of the fold.
struct TBF16 {
    using S = uint16_t;
    using A = float;
    static __device__ __forceinline__ float widen(uint16_t v) {
        return __uint_as_float((uint32_t)v << 16);  // exact
    }
    static __device__ __forceinline__ uint16_t narrow(float f) {
        // v_cvt_pk_bf16_f32: round to nearest even, NaN stays NaN
        return __builtin_bit_cast(uint16_t, (__bf16)f);
    }
};
struct TF32 {
    using S = float;
    using A = float;
    static __device__ __forceinline__ float widen(float v) { return v; }
    static __device__ __forceinline__ float narrow(float f) { return f; }
};
struct TI32 {
    using S = uint32_t;
    using A = uint32_t;  // unsigned: adds wrap modulo 2^32
    static __device__ __forceinline__ uint32_t widen(uint32_t v) { return v; }
    static __device__ __forceinline__ uint32_t narrow(uint32_t v) { return v; }
};

// VE elements in one vector register group; aligned to its size (at most
// 16 bytes) so that it loads as one 8- or 16-byte access per piece.
template <typename S, int VE>
struct alignas(sizeof(S) * VE < 16 ? sizeof(S) * VE : 16) Pack {
    S v[VE];
};

// Tuning knobs (compile time).  Vectors in flight per thread in the ring
// step, and whether streamed operands use non-temporal loads / stores.
#ifndef HOCCL_RS_UNROLL_BF16
#define HOCCL_RS_UNROLL_BF16 2
#endif
#ifndef HOCCL_RS_UNROLL_32
#define HOCCL_RS_UNROLL_32 4
#endif
// Non-temporal access for operands touched once per collective: the ranks'
// inputs (HOCCL_NT_X) and the final output (HOCCL_NT_FINAL).  Partials are
// always accessed normally so that the next step can hit the cache.
#ifndef HOCCL_NT_X
#define HOCCL_NT_X 1
#endif
#ifndef HOCCL_NT_FINAL
#define HOCCL_NT_FINAL 0
#endif
#ifndef HOCCL_FOLD_NT
#define HOCCL_FOLD_NT 1
#endif
#ifndef HOCCL_FOLD_NT_OUT
#define HOCCL_FOLD_NT_OUT 1
#endif
// CU copy: 16-byte vectors in flight per thread and pass, and whether the
// loads and the stores are non-temporal.  Measured on the copy workloads
// (kernel copy path, back to back): 4 vectors with non-temporal stores
// took the FSDP all-gather from 1.08 to 1.02 ms and a 64 MiB copy from 35
// to 31 us against 2 plain vectors, and left the pipeline schedule, the
// EP all-to-all(v) and a 2 GiB copy as they were; non-temporal loads as
// well made the 2 GiB copy 6% faster but the all-gather and the pipeline
// schedule about 20% slower (a shard is read by every rank's copy).
#ifndef HOCCL_COPY_UNROLL
#define HOCCL_COPY_UNROLL 4
#endif
#ifndef HOCCL_COPY_NT_IN
#define HOCCL_COPY_NT_IN 0
#endif
#ifndef HOCCL_COPY_NT_OUT
#define HOCCL_COPY_NT_OUT 1
#endif
// bit 0: in0 non-temporal, bit 1: in1, bit 2: out
constexpr int kNtFirst = (HOCCL_NT_X ? 3 : 0);
constexpr int kNtMiddle = (HOCCL_NT_X ? 2 : 0);
constexpr int kNtLast = (HOCCL_NT_X ? 2 : 0) | (HOCCL_NT_FINAL ? 4 : 0);
constexpr int kNtOnly = (HOCCL_NT_X ? 3 : 0) | (HOCCL_NT_FINAL ? 4 : 0);

// Lane layout of the ring step.  A lane holds VE consecutive elements of
// every operand.  Where bf16 meets fp32 partials, VE = 4: a lane moves 8 B
// of bf16 and 16 B of fp32, so each load or store instruction of a wave
// covers one contiguous span (512 B or 1 KiB).  With VE = 8 the fp32 side
// would take two 16-byte accesses 32 B apart per lane, each instruction
// touching every line of a 2 KiB span half; that layout ran the headline
// reduce-scatter about 5% slower.  bf16-only steps keep 16-byte vectors.
constexpr int kVeBf16Partial = 4;
constexpr int kVeBf16Only = 8;
constexpr int kVe32 = 4;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Vector load / store of a Pack in 16-byte pieces (8 bytes for an 8-byte
// Pack), optionally non-temporal.
template <bool NT, typename P>
__device__ __forceinline__ P ldp(const P *p) {
    static_assert(sizeof(P) == 8 || sizeof(P) % 16 == 0, "Pack must be 8 bytes or a multiple of 16");
    P r;
    if constexpr (sizeof(P) == 8) {
        u32x2 v = NT ? __builtin_nontemporal_load((const u32x2 *)p) : *(const u32x2 *)p;
        __builtin_memcpy(&r, &v, 8);
    } else {
#pragma unroll
        for (int i = 0; i < (int)(sizeof(P) / 16); ++i) {
            u32x4 v = NT ? __builtin_nontemporal_load((const u32x4 *)p + i) : ((const u32x4 *)p)[i];
            __builtin_memcpy((char *)&r + 16 * i, &v, 16);
        }
    }
    return r;
}
template <bool NT, typename P>
__device__ __forceinline__ void stp(P *p, const P &x) {
    if constexpr (sizeof(P) == 8) {
        u32x2 v;
        __builtin_memcpy(&v, &x, 8);
        if (NT)
            __builtin_nontemporal_store(v, (u32x2 *)p);
        else
            *(u32x2 *)p = v;
    } else {
#pragma unroll
        for (int i = 0; i < (int)(sizeof(P) / 16); ++i) {
            u32x4 v;
            __builtin_memcpy(&v, (const char *)&x + 16 * i, 16);
            if (NT)
                __builtin_nontemporal_store(v, (u32x4 *)p + i);
            else
                ((u32x4 *)p)[i] = v;
        }
    }
}

// Splits the blocks of a launch over `nseg` segments.  With at least one
// block per segment, block b serves segment b % nseg (consecutive blocks go
// to different segments, so every XCD streams every segment); otherwise each
// block walks several segments.
template <typename F>
__device__ __forceinline__ void for_each_segment(int nseg, F &&f) {
    if ((int)gridDim.x >= nseg) {
        int seg = (int)blockIdx.x % nseg;
        int lb = (int)blockIdx.x / nseg;
        int nb = ((int)gridDim.x - seg + nseg - 1) / nseg;
        f(seg, lb, nb);
    } else {
        for (int seg = (int)blockIdx.x; seg < nseg; seg += (int)gridDim.x) f(seg, 0, 1);
    }
}

// ---- one ring step --------------------------------------------------------------
template <class T0, class T1, class TO, int VE, int U, int NT>
__device__ __forceinline__ void reduce_segment(const RSegArg &s, int lb, int nb) {
    constexpr bool NT0 = NT & 1, NT1 = NT & 2, NTO = NT & 4;
    using S0 = typename T0::S;
    using S1 = typename T1::S;
    using SO = typename TO::S;
    using P0 = Pack<S0, VE>;
    using P1 = Pack<S1, VE>;
    using PO = Pack<SO, VE>;
    const S0 *in0 = (const S0 *)s.in0;
    const S1 *in1 = (const S1 *)s.in1;
    SO *out = (SO *)s.out;
    const uint64_t n = s.n;

    // Elements before in1 reaches 16-byte alignment; the vector body needs
    // in0, in1 and out all 16-byte aligned at the same element.
    uint64_t h = ((16u - ((uintptr_t)in1 & 15u)) & 15u) / sizeof(S1);
    if (h > n) h = n;
    const bool vec = ((((uintptr_t)(in0 + h)) | ((uintptr_t)(in1 + h)) | ((uintptr_t)(out + h))) &
                      15u) == 0;
    if (!vec) h = n;
    const uint64_t nv = (n - h) / VE;
    const uint64_t tail = h + nv * VE;

    const uint64_t bd = blockDim.x;
    const uint64_t t = (uint64_t)lb * bd + threadIdx.x;
    const uint64_t stride = (uint64_t)nb * bd;
    for (uint64_t k = t; k < h; k += stride)
        out[k] = TO::narrow(T0::widen(in0[k]) + T1::widen(in1[k]));
    for (uint64_t k = tail + t; k < n; k += stride)
        out[k] = TO::narrow(T0::widen(in0[k]) + T1::widen(in1[k]));

    const P0 *v0 = (const P0 *)(in0 + h);
    const P1 *v1 = (const P1 *)(in1 + h);
    PO *vo = (PO *)(out + h);
    auto one = [&](const P0 &a, const P1 &b) {
        PO y;
#pragma unroll
        for (int e = 0; e < VE; ++e) y.v[e] = TO::narrow(T0::widen(a.v[e]) + T1::widen(b.v[e]));
        return y;
    };
    // Main loop: U vectors per thread, all in range, loads issued before use.
    uint64_t base = (uint64_t)lb * bd * U + threadIdx.x;
    for (; base + (uint64_t)(U - 1) * bd < nv; base += stride * U) {
        P0 a[U];
        P1 b[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            a[u] = ldp<NT0>(v0 + base + (uint64_t)u * bd);
            b[u] = ldp<NT1>(v1 + base + (uint64_t)u * bd);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) stp<NTO>(vo + base + (uint64_t)u * bd, one(a[u], b[u]));
    }
    // At most one partial iteration is left for this thread.
#pragma unroll
    for (int u = 0; u < U; ++u) {
        uint64_t i = base + (uint64_t)u * bd;
        if (i < nv) stp<NTO>(vo + i, one(ldp<NT0>(v0 + i), ldp<NT1>(v1 + i)));
    }
}

template <typename A>
__device__ __forceinline__ const A &kernargs();

template <class T0, class T1, class TO, int VE, int U, int NT, int CAP>
__global__ void __launch_bounds__(1024) reduce_step_kernel(ReduceArgsT<CAP>) {
    const ReduceArgsT<CAP> &a = kernargs<ReduceArgsT<CAP>>();
    for_each_segment(a.nseg, [&](int seg, int lb, int nb) {
        reduce_segment<T0, T1, TO, VE, U, NT>(a.seg[seg], lb, nb);
    });
}

// ---- fused ring hops ---------------------------------------------------------------
// One launch folds several consecutive ring hops of every segment: the
// partial (or, on the ring's first hop, the previous rank's own element) is
// loaded once, the nloc contributions are added to it in the ring's order
// while it stays in registers, and the result is stored once.  The adds are
// the ring's adds in the ring's order, so the bits are the ring's; only the
// partial's round trips through memory between the fused hops are gone.
// nloc is the same for every lane, so the guards on the unrolled
// contribution loop are uniform branches.
template <class T0, class T1, class TO, int VE, int U, int NT, int MAXL, bool RH>
__device__ __forceinline__ void multihop_segment(const MSegArg &s, int lb, int nb) {
    constexpr bool NT0 = NT & 1, NT1 = NT & 2, NTO = NT & 4;
    using S0 = typename T0::S;
    using S1 = typename T1::S;
    using SO = typename TO::S;
    using A = typename T1::A;
    // RH: every addition's result is rounded to the contribution's type
    // before the next (bf16 partials), as separate hops would round it.
    auto add = [](A acc, S1 x) -> A {
        A y = acc + T1::widen(x);
        if constexpr (RH) y = T1::widen(T1::narrow(y));
        return y;
    };
    using P0 = Pack<S0, VE>;
    using P1 = Pack<S1, VE>;
    using PO = Pack<SO, VE>;
    const S0 *in0 = (const S0 *)s.in0;
    SO *out = (SO *)s.out;
    const int nl = s.nloc;
    const uint64_t n = s.n;
    const S1 *loc[MAXL];
#pragma unroll
    for (int m = 0; m < MAXL; ++m) loc[m] = m < nl ? (const S1 *)s.loc[m] : (const S1 *)s.loc[0];

    // Elements before the first contribution reaches 16-byte alignment; the
    // vector body needs every operand 16-byte aligned at the same element.
    uint64_t h = ((16u - ((uintptr_t)loc[0] & 15u)) & 15u) / sizeof(S1);
    if (h > n) h = n;
    uintptr_t mis = (uintptr_t)(in0 + h) | (uintptr_t)(out + h);
#pragma unroll
    for (int m = 0; m < MAXL; ++m) mis |= (uintptr_t)(loc[m] + h);
    if (mis & 15u) h = n;
    const uint64_t nv = (n - h) / VE;
    const uint64_t tail = h + nv * VE;

    const uint64_t bd = blockDim.x;
    const uint64_t t = (uint64_t)lb * bd + threadIdx.x;
    const uint64_t stride = (uint64_t)nb * bd;
    auto scalar = [&](uint64_t k) {
        A acc = T0::widen(in0[k]);
#pragma unroll
        for (int m = 0; m < MAXL; ++m)
            if (m < nl) acc = add(acc, loc[m][k]);
        out[k] = TO::narrow(acc);
    };
    for (uint64_t k = t; k < h; k += stride) scalar(k);
    for (uint64_t k = tail + t; k < n; k += stride) scalar(k);

    const P0 *v0 = (const P0 *)(in0 + h);
    const P1 *vl[MAXL];
#pragma unroll
    for (int m = 0; m < MAXL; ++m) vl[m] = (const P1 *)(loc[m] + h);
    PO *vo = (PO *)(out + h);
    auto one = [&](uint64_t i) {
        P0 a = ldp<NT0>(v0 + i);
        P1 b[MAXL];
#pragma unroll
        for (int m = 0; m < MAXL; ++m)
            if (m < nl) b[m] = ldp<NT1>(vl[m] + i);
        A acc[VE];
#pragma unroll
        for (int e = 0; e < VE; ++e) acc[e] = T0::widen(a.v[e]);
#pragma unroll
        for (int m = 0; m < MAXL; ++m)
            if (m < nl)
#pragma unroll
                for (int e = 0; e < VE; ++e) acc[e] = add(acc[e], b[m].v[e]);
        PO y;
#pragma unroll
        for (int e = 0; e < VE; ++e) y.v[e] = TO::narrow(acc[e]);
        stp<NTO>(vo + i, y);
    };
    // Main loop: U vectors of every operand per thread, all in range, every
    // load issued before the adds consume them.
    uint64_t base = (uint64_t)lb * bd * U + threadIdx.x;
    for (; base + (uint64_t)(U - 1) * bd < nv; base += stride * U) {
        P0 a[U];
        P1 b[U][MAXL];
#pragma unroll
        for (int u = 0; u < U; ++u) a[u] = ldp<NT0>(v0 + base + (uint64_t)u * bd);
#pragma unroll
        for (int m = 0; m < MAXL; ++m)
            if (m < nl)
#pragma unroll
                for (int u = 0; u < U; ++u) b[u][m] = ldp<NT1>(vl[m] + base + (uint64_t)u * bd);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            A acc[VE];
#pragma unroll
            for (int e = 0; e < VE; ++e) acc[e] = T0::widen(a[u].v[e]);
#pragma unroll
            for (int m = 0; m < MAXL; ++m)
                if (m < nl)
#pragma unroll
                    for (int e = 0; e < VE; ++e) acc[e] = add(acc[e], b[u][m].v[e]);
            PO y;
#pragma unroll
            for (int e = 0; e < VE; ++e) y.v[e] = TO::narrow(acc[e]);
            stp<NTO>(vo + base + (uint64_t)u * bd, y);
        }
    }
    // At most one partial iteration is left for this thread.
#pragma unroll
    for (int u = 0; u < U; ++u) {
        uint64_t i = base + (uint64_t)u * bd;
        if (i < nv) one(i);
    }
}

template <class T0, class T1, class TO, int VE, int U, int NT, int MAXL, int CAP, bool RH>
__global__ void __launch_bounds__(1024) multihop_kernel(MultiArgsT<CAP>) {
    const MultiArgsT<CAP> &a = kernargs<MultiArgsT<CAP>>();
    for_each_segment(a.nseg, [&](int seg, int lb, int nb) __attribute__((always_inline)) {
        multihop_segment<T0, T1, TO, VE, U, NT, MAXL, RH>(a.seg[seg], lb, nb);
    });
}

// ---- direct fold ------------------------------------------------------------------
// Chunk j reads x[(j+1)%R], x[(j+2)%R], ..., x[j] at the chunk's elements and
// adds them left to right; loads are issued in batches of KB ranks so several
// are in flight before the adds consume them in order.  RH rounds every
// addition's result to the element type before the next addition (the
// partials a ring of bf16 forwarding ranks would hold).
template <class T, int VE, int NR, bool RH, class FA>
__device__ __forceinline__ void fold_chunk(const FA &a, int j, int lb, int nb) {
    using S = typename T::S;
    using A = typename T::A;
    using P = Pack<S, VE>;
    auto add = [](A acc, S x) -> A {
        A y = acc + T::widen(x);
        if constexpr (RH) y = T::widen(T::narrow(y));
        return y;
    };
    const int R = NR > 0 ? NR : a.R;
    const uint64_t e0 = (uint64_t)j * a.c;
    if (e0 >= a.total) return;
    const uint64_t n = (a.total - e0 < a.c) ? a.total - e0 : a.c;
    // k-th operand of chunk j's fold (k = 0 .. R-1) is rank (j + 1 + k) mod R.
    auto src = [&](int k) -> const S * {
        int r = j + 1 + k;
        if (r >= R) r -= R;
        if (r >= R) r -= R;
        return (const S *)a.in[r] + e0;
    };
    const uint64_t oe = a.out_at_chunk ? 0 : e0;
    const int nout = a.write_all ? R : 1;
    auto dst = [&](int q) -> S * { return (S *)a.out[a.write_all ? q : j] + oe; };

    uint64_t h = ((16u - ((uintptr_t)src(0) & 15u)) & 15u) / sizeof(S);
    if (h > n) h = n;
    uintptr_t mis = 0;
    for (int k = 0; k < R; ++k) mis |= (uintptr_t)(src(k) + h);
    for (int q = 0; q < nout; ++q) mis |= (uintptr_t)(dst(q) + h);
    if (mis & 15u) h = n;
    const uint64_t nv = (n - h) / VE;
    const uint64_t tail = h + nv * VE;

    const uint64_t bd = blockDim.x;
    const uint64_t t = (uint64_t)lb * bd + threadIdx.x;
    const uint64_t stride = (uint64_t)nb * bd;
    auto scalar = [&](uint64_t k) {
        A acc = T::widen(src(0)[k]);
        for (int q = 1; q < R; ++q) acc = add(acc, src(q)[k]);
        S y = T::narrow(acc);
        for (int q = 0; q < nout; ++q) dst(q)[k] = y;
    };
    for (uint64_t k = t; k < h; k += stride) scalar(k);
    for (uint64_t k = tail + t; k < n; k += stride) scalar(k);

    constexpr bool NT = HOCCL_FOLD_NT;
    constexpr bool NTO = HOCCL_FOLD_NT_OUT;
    if constexpr (NR > 0) {
        // The operand and output pointers are computed once, outside the
        // loop; every operand's vector is loaded before the in-order adds
        // consume them.  Reading an output pointer from the argument buffer
        // inside the loop put a scalar load and its wait in front of every
        // store (about 7% of the headline fold's time).
        const P *sp[NR];
#pragma unroll
        for (int k = 0; k < NR; ++k) sp[k] = (const P *)(src(k) + h);
        auto run = [&](auto outs) {
            constexpr int NO = decltype(outs)::value;
            P *dp[NO];
#pragma unroll
            for (int q = 0; q < NO; ++q) dp[q] = (P *)(dst(q) + h);
            for (uint64_t i = t; i < nv; i += stride) {
                P v[NR];
#pragma unroll
                for (int k = 0; k < NR; ++k) v[k] = ldp<NT>(sp[k] + i);
                A acc[VE];
#pragma unroll
                for (int e = 0; e < VE; ++e) acc[e] = T::widen(v[0].v[e]);
#pragma unroll
                for (int k = 1; k < NR; ++k)
#pragma unroll
                    for (int e = 0; e < VE; ++e) acc[e] = add(acc[e], v[k].v[e]);
                P y;
#pragma unroll
                for (int e = 0; e < VE; ++e) y.v[e] = T::narrow(acc[e]);
#pragma unroll
                for (int q = 0; q < NO; ++q) stp<NTO>(dp[q] + i, y);
            }
        };
        if (a.write_all)
            run(std::integral_constant<int, NR>{});
        else
            run(std::integral_constant<int, 1>{});
        return;
    }
    for (uint64_t i = t; i < nv; i += stride) {
        A acc[VE];
        {
            constexpr int KB = 8;
            {
                P v0 = ((const P *)(src(0) + h))[i];
#pragma unroll
                for (int e = 0; e < VE; ++e) acc[e] = T::widen(v0.v[e]);
            }
            int k = 1;
            for (; k + KB <= R; k += KB) {
                P v[KB];
#pragma unroll
                for (int q = 0; q < KB; ++q) v[q] = ((const P *)(src(k + q) + h))[i];
#pragma unroll
                for (int q = 0; q < KB; ++q)
#pragma unroll
                    for (int e = 0; e < VE; ++e) acc[e] = add(acc[e], v[q].v[e]);
            }
            for (; k < R; ++k) {
                P v = ((const P *)(src(k) + h))[i];
#pragma unroll
                for (int e = 0; e < VE; ++e) acc[e] = add(acc[e], v.v[e]);
            }
        }
        P y;
#pragma unroll
        for (int e = 0; e < VE; ++e) y.v[e] = T::narrow(acc[e]);
        for (int q = 0; q < nout; ++q) ((P *)(dst(q) + h))[i] = y;
    }
}

// The argument structs are indexed with run-time rank numbers.  Reading them
// through the kernarg segment pointer keeps those reads scalar loads from the
// (read-only) argument buffer; indexing the by-value parameter instead makes
// the compiler copy the whole struct into per-thread scratch memory.
template <typename A>
__device__ __forceinline__ const A &kernargs() {
    return *(const A *)__builtin_amdgcn_kernarg_segment_ptr();
}

template <class T, int VE, int NR, int CAP, bool RH>
__global__ void __launch_bounds__(1024) fold_kernel(FoldArgsT<CAP>) {
    const FoldArgsT<CAP> &a = kernargs<FoldArgsT<CAP>>();
    // Forced inline: for_each_segment calls the body from two places, and
    // the eight-rank rounding fold was otherwise left an out-of-line call
    // with a scratch frame.
    for_each_segment(a.R, [&](int j, int lb, int nb) __attribute__((always_inline)) {
        fold_chunk<T, VE, NR, RH>(a, j, lb, nb);
    });
}

// ---- CU copy ----------------------------------------------------------------------
template <int U>
__device__ __forceinline__ void copy_segment(const CSegArg &s, int lb, int nb) {
    const unsigned char *src = (const unsigned char *)s.src;
    unsigned char *dst = (unsigned char *)s.dst;
    const uint64_t n = s.bytes;
    const uint64_t bd = blockDim.x;
    const uint64_t t = (uint64_t)lb * bd + threadIdx.x;
    const uint64_t stride = (uint64_t)nb * bd;
    // Widest unit for which source and destination share their misalignment.
    const uintptr_t x = (uintptr_t)src ^ (uintptr_t)dst;
    const uint64_t w = (x & 15u) == 0 ? 16 : ((x & 3u) == 0 ? 4 : 1);
    uint64_t h = w == 1 ? 0 : ((w - ((uintptr_t)src & (w - 1))) & (w - 1));
    if (h > n) h = n;
    const uint64_t nv = w == 1 ? 0 : (n - h) / w;
    const uint64_t tail = h + nv * w;
    for (uint64_t k = t; k < h; k += stride) dst[k] = src[k];
    for (uint64_t k = (w == 1 ? 0 : tail) + t; k < n; k += stride) dst[k] = src[k];
    if (w == 16) {
        using V = Pack<uint32_t, 4>;  // HIP's uint4 is a union and defeats SROA
        const V *vs = (const V *)(src + h);
        V *vd = (V *)(dst + h);
        uint64_t base = (uint64_t)lb * bd * U + threadIdx.x;
        for (; base + (uint64_t)(U - 1) * bd < nv; base += stride * U) {
            V v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = ldp<HOCCL_COPY_NT_IN>(vs + base + (uint64_t)u * bd);
#pragma unroll
            for (int u = 0; u < U; ++u) stp<HOCCL_COPY_NT_OUT>(vd + base + (uint64_t)u * bd, v[u]);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            uint64_t i = base + (uint64_t)u * bd;
            if (i < nv) vd[i] = vs[i];
        }
    } else if (w == 4) {
        const uint32_t *vs = (const uint32_t *)(src + h);
        uint32_t *vd = (uint32_t *)(dst + h);
        for (uint64_t i = t; i < nv; i += stride) vd[i] = vs[i];
    }
}

constexpr int kCopyUnroll = HOCCL_COPY_UNROLL;

template <int CAP>
__global__ void __launch_bounds__(1024) copy_kernel(CopyArgsT<CAP>) {
    const CopyArgsT<CAP> &a = kernargs<CopyArgsT<CAP>>();
    for_each_segment(a.nseg, [&](int seg, int lb, int nb) {
        copy_segment<kCopyUnroll>(a.seg[seg], lb, nb);
    });
}

}  // namespace

// ---- launchers --------------------------------------------------------------------

// hipLaunchKernel reports this launch's own status (hipGetLastError would
// also return errors left behind by unrelated earlier calls).
template <typename Args>
static hipError_t launch(const void *kernel, const Args &a, int wg, int threads, hipStream_t s) {
    void *args[] = {const_cast<Args *>(&a)};
    return hipLaunchKernel(kernel, dim3((unsigned)wg), dim3((unsigned)threads), args, 0, s);
}

// The first a.nseg slots of `a` in an argument struct of CAP slots.
template <int CAP>
static ReduceArgsT<CAP> fit(const ReduceArgs &a) {
    ReduceArgsT<CAP> b{};
    for (int k = 0; k < a.nseg; ++k) b.seg[k] = a.seg[k];
    b.nseg = a.nseg;
    return b;
}
template <int CAP>
static MultiArgsT<CAP> fit(const MultiArgs &a) {
    MultiArgsT<CAP> b{};
    for (int k = 0; k < a.nseg; ++k) b.seg[k] = a.seg[k];
    b.nseg = a.nseg;
    return b;
}
template <int CAP>
static CopyArgsT<CAP> fit(const CopyArgs &a) {
    CopyArgsT<CAP> b{};
    for (int k = 0; k < a.nseg; ++k) b.seg[k] = a.seg[k];
    b.nseg = a.nseg;
    return b;
}
template <int CAP>
static FoldArgsT<CAP> fit(const FoldArgs &a) {
    FoldArgsT<CAP> b{};
    for (int r = 0; r < a.R; ++r) {
        b.in[r] = a.in[r];
        b.out[r] = a.out[r];
    }
    b.c = a.c;
    b.total = a.total;
    b.R = a.R;
    b.write_all = a.write_all;
    b.out_at_chunk = a.out_at_chunk;
    return b;
}

// Ring steps of up to 8 ranks (264 bytes of arguments) or up to 64 (2 KiB).
constexpr int kSmallSegs = 8;

template <class T0, class T1, class TO, int VE, int U, int NT>
static hipError_t launch_rs(const ReduceArgs &a, int wg, int threads, hipStream_t s) {
    if (a.nseg <= kSmallSegs)
        return launch((const void *)reduce_step_kernel<T0, T1, TO, VE, U, NT, kSmallSegs>,
                      fit<kSmallSegs>(a), wg, threads, s);
    return launch((const void *)reduce_step_kernel<T0, T1, TO, VE, U, NT, kMaxReduceSegs>, a, wg,
                  threads, s);
}

hipError_t launch_reduce_step(hoccl_dtype_t dt, Phase ph, const ReduceArgs &a, int wg, int threads,
                              hipStream_t s, bool bf16_partials) {
    constexpr int UB = HOCCL_RS_UNROLL_BF16, U4 = HOCCL_RS_UNROLL_32;
    constexpr int VP = kVeBf16Partial, VB = kVeBf16Only, V4 = kVe32;
    if (dt == HOCCL_BF16 && bf16_partials) {
        // Every operand and result in bf16: each step rounds its sum, as a
        // ring that forwards bf16 partials does.  The same in-flight rule
        // as below, on 8-element vectors.
        uint64_t n = 0;
        for (int k = 0; k < a.nseg; ++k) n += a.seg[k].n;
        const bool deep = n > (uint64_t)wg * (uint64_t)threads * (uint64_t)(VB * UB);
        if (deep) {
            switch (ph) {
            case PH_FIRST: return launch_rs<TBF16, TBF16, TBF16, VB, 2 * UB, kNtFirst>(a, wg, threads, s);
            case PH_MIDDLE: return launch_rs<TBF16, TBF16, TBF16, VB, 2 * UB, kNtMiddle>(a, wg, threads, s);
            case PH_LAST: return launch_rs<TBF16, TBF16, TBF16, VB, 2 * UB, kNtLast>(a, wg, threads, s);
            case PH_ONLY: break;
            }
        }
        switch (ph) {
        case PH_FIRST: return launch_rs<TBF16, TBF16, TBF16, VB, UB, kNtFirst>(a, wg, threads, s);
        case PH_MIDDLE: return launch_rs<TBF16, TBF16, TBF16, VB, UB, kNtMiddle>(a, wg, threads, s);
        case PH_LAST: return launch_rs<TBF16, TBF16, TBF16, VB, UB, kNtLast>(a, wg, threads, s);
        case PH_ONLY: return launch_rs<TBF16, TBF16, TBF16, VB, UB, kNtOnly>(a, wg, threads, s);
        }
    } else if (dt == HOCCL_BF16) {
        // A launch that leaves each thread several passes (a small
        // workgroup budget) keeps twice the vectors in flight per thread:
        // there the bytes in flight per wave, not the number of waves, set
        // the rate (8 workgroups: 777 us per headline step with 2 vectors,
        // 497 us with 4).
        uint64_t n = 0;
        for (int k = 0; k < a.nseg; ++k) n += a.seg[k].n;
        const bool deep = n > (uint64_t)wg * (uint64_t)threads * (uint64_t)(VP * UB);
        if (deep) {
            switch (ph) {
            case PH_FIRST: return launch_rs<TBF16, TBF16, TF32, VP, 2 * UB, kNtFirst>(a, wg, threads, s);
            case PH_MIDDLE: return launch_rs<TF32, TBF16, TF32, VP, 2 * UB, kNtMiddle>(a, wg, threads, s);
            case PH_LAST: return launch_rs<TF32, TBF16, TBF16, VP, 2 * UB, kNtLast>(a, wg, threads, s);
            case PH_ONLY: return launch_rs<TBF16, TBF16, TBF16, VB, UB, kNtOnly>(a, wg, threads, s);
            }
        }
        switch (ph) {
        case PH_FIRST: return launch_rs<TBF16, TBF16, TF32, VP, UB, kNtFirst>(a, wg, threads, s);
        case PH_MIDDLE: return launch_rs<TF32, TBF16, TF32, VP, UB, kNtMiddle>(a, wg, threads, s);
        case PH_LAST: return launch_rs<TF32, TBF16, TBF16, VP, UB, kNtLast>(a, wg, threads, s);
        case PH_ONLY: return launch_rs<TBF16, TBF16, TBF16, VB, UB, kNtOnly>(a, wg, threads, s);
        }
    } else if (dt == HOCCL_FP32) {
        switch (ph) {
        case PH_FIRST: return launch_rs<TF32, TF32, TF32, V4, U4, kNtFirst>(a, wg, threads, s);
        case PH_MIDDLE: return launch_rs<TF32, TF32, TF32, V4, U4, kNtMiddle>(a, wg, threads, s);
        case PH_LAST: return launch_rs<TF32, TF32, TF32, V4, U4, kNtLast>(a, wg, threads, s);
        case PH_ONLY: return launch_rs<TF32, TF32, TF32, V4, U4, kNtOnly>(a, wg, threads, s);
        }
    } else if (dt == HOCCL_INT32) {
        switch (ph) {
        case PH_FIRST: return launch_rs<TI32, TI32, TI32, V4, U4, kNtFirst>(a, wg, threads, s);
        case PH_MIDDLE: return launch_rs<TI32, TI32, TI32, V4, U4, kNtMiddle>(a, wg, threads, s);
        case PH_LAST: return launch_rs<TI32, TI32, TI32, V4, U4, kNtLast>(a, wg, threads, s);
        case PH_ONLY: return launch_rs<TI32, TI32, TI32, V4, U4, kNtOnly>(a, wg, threads, s);
        }
    }
    return hipErrorInvalidValue;
}

// Fused ring hops.  Every lane moves 4 elements of every operand (8 bytes of
// bf16, 16 of fp32 / int32), and keeps U such vectors of each operand in
// flight, U chosen per bound on the contributions so that the registers
// they need stay within the 128 VGPRs a 1024-thread launch bound allows
// without spilling: bf16 2 whatever the bound; 32-bit types 4, 2 and 1 for
// at most 2, 4 and 8 contributions.
template <class T0, class T1, class TO, int NT, int MAXL, bool RH>
static hipError_t launch_mh_l(const MultiArgs &a, int wg, int threads, hipStream_t s) {
    constexpr int U = sizeof(typename T1::S) == 2 ? 2 : (MAXL <= 2 ? 4 : (MAXL <= 4 ? 2 : 1));
    if (a.nseg <= kSmallSegs)
        return launch((const void *)multihop_kernel<T0, T1, TO, 4, U, NT, MAXL, kSmallSegs, RH>,
                      fit<kSmallSegs>(a), wg, threads, s);
    return launch((const void *)multihop_kernel<T0, T1, TO, 4, U, NT, MAXL, kMaxMultiSegs, RH>, a, wg,
                  threads, s);
}

template <class T0, class T1, class TO, int NT, bool RH = false>
static hipError_t launch_mh(const MultiArgs &a, int wg, int threads, hipStream_t s) {
    int nl = 0;
    for (int k = 0; k < a.nseg; ++k) nl = a.seg[k].nloc > nl ? a.seg[k].nloc : nl;
    if (nl <= 2) return launch_mh_l<T0, T1, TO, NT, 2, RH>(a, wg, threads, s);
    if (nl <= 4) return launch_mh_l<T0, T1, TO, NT, 4, RH>(a, wg, threads, s);
    return launch_mh_l<T0, T1, TO, NT, kMaxHops, RH>(a, wg, threads, s);
}

hipError_t launch_multihop(hoccl_dtype_t dt, Phase ph, const MultiArgs &a, int wg, int threads,
                           hipStream_t s, bool bf16_partials) {
    if (dt == HOCCL_BF16 && bf16_partials) {
        switch (ph) {
        case PH_FIRST: return launch_mh<TBF16, TBF16, TBF16, kNtFirst, true>(a, wg, threads, s);
        case PH_MIDDLE: return launch_mh<TBF16, TBF16, TBF16, kNtMiddle, true>(a, wg, threads, s);
        case PH_LAST: return launch_mh<TBF16, TBF16, TBF16, kNtLast, true>(a, wg, threads, s);
        case PH_ONLY: return launch_mh<TBF16, TBF16, TBF16, kNtOnly, true>(a, wg, threads, s);
        }
    } else if (dt == HOCCL_BF16) {
        switch (ph) {
        case PH_FIRST: return launch_mh<TBF16, TBF16, TF32, kNtFirst>(a, wg, threads, s);
        case PH_MIDDLE: return launch_mh<TF32, TBF16, TF32, kNtMiddle>(a, wg, threads, s);
        case PH_LAST: return launch_mh<TF32, TBF16, TBF16, kNtLast>(a, wg, threads, s);
        case PH_ONLY: return launch_mh<TBF16, TBF16, TBF16, kNtOnly>(a, wg, threads, s);
        }
    } else if (dt == HOCCL_FP32) {
        switch (ph) {
        case PH_FIRST: return launch_mh<TF32, TF32, TF32, kNtFirst>(a, wg, threads, s);
        case PH_MIDDLE: return launch_mh<TF32, TF32, TF32, kNtMiddle>(a, wg, threads, s);
        case PH_LAST: return launch_mh<TF32, TF32, TF32, kNtLast>(a, wg, threads, s);
        case PH_ONLY: return launch_mh<TF32, TF32, TF32, kNtOnly>(a, wg, threads, s);
        }
    } else if (dt == HOCCL_INT32) {
        switch (ph) {
        case PH_FIRST: return launch_mh<TI32, TI32, TI32, kNtFirst>(a, wg, threads, s);
        case PH_MIDDLE: return launch_mh<TI32, TI32, TI32, kNtMiddle>(a, wg, threads, s);
        case PH_LAST: return launch_mh<TI32, TI32, TI32, kNtLast>(a, wg, threads, s);
        case PH_ONLY: return launch_mh<TI32, TI32, TI32, kNtOnly>(a, wg, threads, s);
        }
    }
    return hipErrorInvalidValue;
}

// Grid sizing for fused launches assumes 2 vectors of 4 elements per pass.
size_t multihop_elems_per_thread(hoccl_dtype_t) { return 8; }

// Elements one thread covers in one pass of each kernel's main loop; the
// executor sizes automatic launches to about one pass per thread.
size_t reduce_step_elems_per_thread(hoccl_dtype_t dt, Phase ph, bool bf16_partials) {
    if (dt == HOCCL_BF16)
        return (size_t)(ph == PH_ONLY || bf16_partials ? kVeBf16Only : kVeBf16Partial) *
               HOCCL_RS_UNROLL_BF16;
    return (size_t)kVe32 * HOCCL_RS_UNROLL_32;
}
size_t fold_elems_per_thread(hoccl_dtype_t dt) { return 16 / dtype_size(dt); }
size_t copy_bytes_per_thread() { return 16 * kCopyUnroll; }

// R = 2, 3, 4 and 8 have kernels of their own, whose arguments hold R ranks.
template <class T, int VE, int NR, bool RH>
static hipError_t launch_fold_r(const FoldArgs &a, int wg, int threads, hipStream_t s) {
    return launch((const void *)fold_kernel<T, VE, NR, NR, RH>, fit<NR>(a), wg, threads, s);
}

template <class T, int VE, bool RH = false>
static hipError_t launch_fold_t(const FoldArgs &a, int wg, int threads, hipStream_t s) {
    switch (a.R) {
    case 2: return launch_fold_r<T, VE, 2, RH>(a, wg, threads, s);
    case 3: return launch_fold_r<T, VE, 3, RH>(a, wg, threads, s);
    case 4: return launch_fold_r<T, VE, 4, RH>(a, wg, threads, s);
    case 8: return launch_fold_r<T, VE, 8, RH>(a, wg, threads, s);
    default: return launch((const void *)fold_kernel<T, VE, 0, kMaxRanks, RH>, a, wg, threads, s);
    }
}

hipError_t launch_fold(hoccl_dtype_t dt, const FoldArgs &a, int wg, int threads, hipStream_t s,
                       bool bf16_partials) {
    if (dt == HOCCL_BF16 && bf16_partials) return launch_fold_t<TBF16, 8, true>(a, wg, threads, s);
    if (dt == HOCCL_BF16) return launch_fold_t<TBF16, 8>(a, wg, threads, s);
    if (dt == HOCCL_FP32) return launch_fold_t<TF32, 4>(a, wg, threads, s);
    if (dt == HOCCL_INT32) return launch_fold_t<TI32, 4>(a, wg, threads, s);
    return hipErrorInvalidValue;
}

// Copy launches of up to 8, 32 or 128 segments (200 bytes to 3 KiB of arguments).
hipError_t launch_copy(const CopyArgs &a, int wg, int threads, hipStream_t s) {
    if (a.nseg <= 8) return launch((const void *)copy_kernel<8>, fit<8>(a), wg, threads, s);
    if (a.nseg <= 32) return launch((const void *)copy_kernel<32>, fit<32>(a), wg, threads, s);
    return launch((const void *)copy_kernel<kMaxCopySegs>, a, wg, threads, s);
}

}  // namespace hoccl
