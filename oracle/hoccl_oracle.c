/*
 * hoccl_oracle.c -- plain, single-threaded CPU oracle for the collectives of
 * the HOCCL hot path (ring reduce-scatter, all-gather, all-reduce,
 * point-to-point send/recv, all-to-all(v)).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, table or helper with
 * the HIP library; it includes only the C standard library.
 *
 * What each function computes, and where the definition comes from:
 *
 *  - Copy collectives (all-gather, send/recv, all-to-all, all-to-all(v)) are
 *    the data movement the paper describes for background traffic: a
 *    collective is a traffic matrix C of logical flows C[u,v] from GPU u to
 *    GPU v (Collective Scheduler, "Traffic matrix abstraction"), realised as
 *    point-to-point copies (Zero-SM Point-to-Point Executor).  The oracle
 *    writes each flow out as a plain element loop.
 *
 *  - Reductions are explicitly outside the paper's scope (Limitations: the
 *    paper leaves AllReduce and ReduceScatter to SM-side execution).  Their
 *    semantics here are the reading this library adopts:
 *      * the only operator is sum;
 *      * ring direction r -> r+1, and the fold for chunk j starts at rank
 *        j+1 and ends at rank j, so rank j owns the reduced chunk j:
 *            ring_sum(j, i) = ((x[j+1][i] + x[j+2][i]) + ...) + x[j][i]
 *        with rank indices taken mod R;
 *      * int32 adds wrap modulo 2^32;
 *      * fp32 adds are single IEEE binary32 additions, round to nearest even;
 *      * bf16 operands are widened exactly to fp32, all additions are fp32,
 *        and one round-to-nearest-even fp32 -> bf16 conversion happens at
 *        the end (fp32 accumulation);
 *      * a second bf16 mode (the *_bf16_hops functions) passes bf16
 *        partials from hop to hop: every partial is rounded to bf16 right
 *        after its fp32 add, so R ranks round R-1 times (fewer bytes per
 *        hop, more rounding error);
 *      * copies also take bytes (OR_UINT8); the sums refuse them;
 *      * all-reduce splits count n into R chunks of c = ceil(n/R) elements,
 *        chunk j = [j*c, min(n, (j+1)*c)), so the last chunks may be short or
 *        empty;
 *      * reduce-scatter with recvcount n gives rank r block r of the
 *        all-reduce of R*n elements, which therefore equals the matching
 *        slice of the all-reduce bit for bit.
 *
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off -fPIC -shared.  On x86-64
 * float arithmetic is SSE binary32 with the default MXCSR (no flush to zero,
 * no denormals-are-zero), so every float add below is one IEEE add.
 *
 * Every function returns 0 on success and a negative value on an argument
 * error; none allocates memory.
 */
#include <stddef.h>
#include <stdint.h>
#include <string.h>

/* OR_UINT8 is a byte, for the copies only: the sum is defined for the
 * three arithmetic types, so the reductions refuse it. */
enum { OR_INT32 = 0, OR_FP32 = 1, OR_BF16 = 2, OR_UINT8 = 3 };

static size_t elem_size(int dtype)
{
    switch (dtype) {
    case OR_INT32: return 4;
    case OR_FP32: return 4;
    case OR_BF16: return 2;
    case OR_UINT8: return 1;
    default: return 0;
    }
}

/* ---- bf16 <-> fp32, written from the IEEE-754 definitions ---------------- */

/* bf16 is the upper 16 bits of a binary32 value, so widening is exact. */
static float bf16_to_f32(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* Round a binary32 value to bf16, round to nearest, ties to even.  The 16
 * dropped bits are compared with the half-way point 0x8000; at exactly the
 * half-way point the kept part rounds up only when its last bit is 1.  A
 * carry out of the mantissa correctly bumps the exponent, and the largest
 * finite values round to infinity.  NaN keeps its sign and upper payload and
 * gets the quiet bit set, so it never turns into infinity. */
uint16_t oracle_f32_to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu) != 0)
        return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t kept = u >> 16;
    uint32_t dropped = u & 0xffffu;
    if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u)))
        kept += 1u;
    return (uint16_t)kept;
}

void oracle_f32_to_bf16_array(const float *src, uint16_t *dst, size_t n)
{
    for (size_t i = 0; i < n; ++i)
        dst[i] = oracle_f32_to_bf16(src[i]);
}

/* ---- the ring fold --------------------------------------------------------
 * Reduces element i over all R ranks, starting at rank (j+1) mod R and ending
 * at rank j, and stores the result (converted to dtype) into *out. */
static void ring_sum_one(const void *const *x, int dtype, int R, int j,
                         size_t i, void *out)
{
    if (dtype == OR_INT32) {
        uint32_t acc = 0;
        for (int k = 1; k <= R; ++k) {
            const int32_t *xr = (const int32_t *)x[(j + k) % R];
            uint32_t v = (uint32_t)xr[i];
            acc = (k == 1) ? v : acc + v;
        }
        *(int32_t *)out = (int32_t)acc;
    } else if (dtype == OR_FP32) {
        float acc = 0.0f;
        for (int k = 1; k <= R; ++k) {
            const float *xr = (const float *)x[(j + k) % R];
            acc = (k == 1) ? xr[i] : acc + xr[i];
        }
        *(float *)out = acc;
    } else {
        float acc = 0.0f;
        for (int k = 1; k <= R; ++k) {
            const uint16_t *xr = (const uint16_t *)x[(j + k) % R];
            float v = bf16_to_f32(xr[i]);
            acc = (k == 1) ? v : acc + v;
        }
        *(uint16_t *)out = oracle_f32_to_bf16(acc);
    }
}

/* The same fold with bf16 partials: the partial is rounded to bf16 (round to
 * nearest, ties to even) after every add, as when each hop passes a bf16
 * partial to the next rank.  Two ranks need one add and one rounding, the
 * same as the fold above. */
static uint16_t ring_sum_one_bf16_hops(const void *const *x, int R, int j, size_t i)
{
    uint16_t part = ((const uint16_t *)x[(j + 1) % R])[i];
    for (int k = 2; k <= R; ++k) {
        const uint16_t *xr = (const uint16_t *)x[(j + k) % R];
        part = oracle_f32_to_bf16(bf16_to_f32(part) + bf16_to_f32(xr[i]));
    }
    return part;
}

static int check_common(const void *send, const void *recv, int dtype, int R)
{
    if (R < 1 || R > 64) return -1;
    if (elem_size(dtype) == 0) return -2;
    if (!send || !recv) return -3;
    return 0;
}

/* all-reduce: every rank receives the ring sum of all R inputs; element i
 * belongs to chunk floor(i / ceil(count / R)). */
int oracle_allreduce(const void *const *send, void *const *recv, size_t count,
                     int dtype, int R)
{
    int rc = check_common(send, recv, dtype, R);
    if (rc) return rc;
    if (dtype == OR_UINT8) return -2;
    if (count == 0) return 0;
    size_t es = elem_size(dtype);
    size_t c = (count + (size_t)R - 1) / (size_t)R;
    for (size_t i = 0; i < count; ++i) {
        unsigned char v[4];
        ring_sum_one(send, dtype, R, (int)(i / c), i, v);
        for (int r = 0; r < R; ++r)
            memcpy((unsigned char *)recv[r] + i * es, v, es);
    }
    return 0;
}

/* reduce-scatter: each send buffer holds R*recvcount elements; rank r
 * receives block r of the ring sum, whose fold ends at rank r. */
int oracle_reduce_scatter(const void *const *send, void *const *recv,
                          size_t recvcount, int dtype, int R)
{
    int rc = check_common(send, recv, dtype, R);
    if (rc) return rc;
    if (dtype == OR_UINT8) return -2;
    size_t es = elem_size(dtype);
    for (int r = 0; r < R; ++r)
        for (size_t i = 0; i < recvcount; ++i)
            ring_sum_one(send, dtype, R, r, (size_t)r * recvcount + i,
                         (unsigned char *)recv[r] + i * es);
    return 0;
}

/* all-gather: recv_r[s*n + i] = x_s[i] for every r, bitwise. */
int oracle_allgather(const void *const *send, void *const *recv,
                     size_t sendcount, int dtype, int R)
{
    int rc = check_common(send, recv, dtype, R);
    if (rc) return rc;
    size_t es = elem_size(dtype);
    for (int r = 0; r < R; ++r)
        for (int s = 0; s < R; ++s)
            for (size_t i = 0; i < sendcount; ++i)
                memcpy((unsigned char *)recv[r] + ((size_t)s * sendcount + i) * es,
                       (const unsigned char *)send[s] + i * es, es);
    return 0;
}

/* send/recv: rank r with peers[r] = d >= 0 sends its count elements to rank
 * d.  A receiver named twice is an error; receivers nobody sends to are left
 * untouched. */
int oracle_sendrecv(const void *const *send, void *const *recv,
                    const int *peers, size_t count, int dtype, int R)
{
    int rc = check_common(send, recv, dtype, R);
    if (rc) return rc;
    if (!peers) return -3;
    unsigned char seen[64];
    memset(seen, 0, sizeof seen);
    for (int r = 0; r < R; ++r) {
        int d = peers[r];
        if (d < -1 || d >= R) return -4;
        if (d >= 0) {
            if (seen[d]) return -5;
            seen[d] = 1;
        }
    }
    size_t es = elem_size(dtype);
    for (int r = 0; r < R; ++r) {
        int d = peers[r];
        if (d < 0) continue;
        for (size_t i = 0; i < count; ++i)
            memcpy((unsigned char *)recv[d] + i * es,
                   (const unsigned char *)send[r] + i * es, es);
    }
    return 0;
}

/* all-to-all: block d of rank s's send buffer lands in block s of rank d's
 * receive buffer: recv_d[s*n + i] = x_s[d*n + i]. */
int oracle_alltoall(const void *const *send, void *const *recv, size_t count,
                    int dtype, int R)
{
    int rc = check_common(send, recv, dtype, R);
    if (rc) return rc;
    size_t es = elem_size(dtype);
    for (int s = 0; s < R; ++s)
        for (int d = 0; d < R; ++d)
            for (size_t i = 0; i < count; ++i)
                memcpy((unsigned char *)recv[d] + ((size_t)s * count + i) * es,
                       (const unsigned char *)send[s] + ((size_t)d * count + i) * es,
                       es);
    return 0;
}

/* all-to-all(v): the traffic matrix C[s][d] = sendcounts[s*R + d] elements
 * move from x_s at sdispls[s*R + d] to recv_d at rdispls[s*R + d]. */
int oracle_alltoallv(const void *const *send, const size_t *sendcounts,
                     const size_t *sdispls, void *const *recv,
                     const size_t *rdispls, int dtype, int R)
{
    int rc = check_common(send, recv, dtype, R);
    if (rc) return rc;
    if (!sendcounts || !sdispls || !rdispls) return -3;
    size_t es = elem_size(dtype);
    for (int s = 0; s < R; ++s)
        for (int d = 0; d < R; ++d) {
            size_t k = (size_t)s * (size_t)R + (size_t)d;
            for (size_t i = 0; i < sendcounts[k]; ++i)
                memcpy((unsigned char *)recv[d] + (rdispls[k] + i) * es,
                       (const unsigned char *)send[s] + (sdispls[k] + i) * es,
                       es);
        }
    return 0;
}

/* all-reduce and reduce-scatter of bf16 with bf16 partials rounded at every
 * hop (ring_sum_one_bf16_hops), in the ring order and chunking of
 * oracle_allreduce / oracle_reduce_scatter. */
int oracle_allreduce_bf16_hops(const void *const *send, void *const *recv, size_t count, int R)
{
    int rc = check_common(send, recv, OR_BF16, R);
    if (rc) return rc;
    if (count == 0) return 0;
    size_t c = (count + (size_t)R - 1) / (size_t)R;
    for (size_t i = 0; i < count; ++i) {
        uint16_t v = ring_sum_one_bf16_hops(send, R, (int)(i / c), i);
        for (int r = 0; r < R; ++r)
            ((uint16_t *)recv[r])[i] = v;
    }
    return 0;
}

int oracle_reduce_scatter_bf16_hops(const void *const *send, void *const *recv, size_t recvcount, int R)
{
    int rc = check_common(send, recv, OR_BF16, R);
    if (rc) return rc;
    for (int r = 0; r < R; ++r)
        for (size_t i = 0; i < recvcount; ++i)
            ((uint16_t *)recv[r])[i] = ring_sum_one_bf16_hops(send, R, r, (size_t)r * recvcount + i);
    return 0;
}
