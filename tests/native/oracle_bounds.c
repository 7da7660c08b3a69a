/* The CPU oracle under AddressSanitizer and UBSan: every function on buffers
 * of exactly the documented size (each its own allocation), over rank counts
 * 1..64, ragged counts, all dtypes (bytes for the copies, and refused by
 * the sums), and int32 inputs near the wrap-around
 * (signed overflow in the oracle's integer path would be reported).  Values
 * are checked elsewhere; this is about bounds and undefined behaviour.  The
 * oracle is compiled into this file; nothing of the library is. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../oracle/hoccl_oracle.c"

static uint64_t rng = 0x9e3779b97f4a7c15ull;
static uint32_t next32(void)
{
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return (uint32_t)(rng >> 11);
}

static void *fill(size_t bytes, int dtype)
{
    unsigned char *p = malloc(bytes ? bytes : 1);
    size_t es = elem_size(dtype);
    for (size_t i = 0; i + es <= bytes; i += es) {
        uint32_t v = next32();
        if (dtype == 0) v = (v & 1) ? 0x7ffffff0u + (v & 15) : 0x80000000u + (v & 15);
        memcpy(p + i, &v, es);
    }
    return p;
}

static int checked = 0;

static void run_case(int op, int dtype, int R, size_t n)
{
    size_t es = elem_size(dtype);
    void *send[64], *recv[64];
    size_t sb = n * es, rb = n * es;
    if (op == 1 || op == 4) sb = (size_t)R * n * es;   /* reduce-scatter, all-to-all in */
    if (op == 2 || op == 4) rb = (size_t)R * n * es;   /* all-gather, all-to-all out    */
    for (int r = 0; r < R; ++r) {
        send[r] = fill(sb, dtype);
        recv[r] = fill(rb, dtype);
    }
    int rc = 0;
    if (op == 0) rc = oracle_allreduce((const void *const *)send, recv, n, dtype, R);
    if (op == 1) rc = oracle_reduce_scatter((const void *const *)send, recv, n, dtype, R);
    if (op == 2) rc = oracle_allgather((const void *const *)send, recv, n, dtype, R);
    if (op == 3) {
        int peers[64];
        for (int r = 0; r < R; ++r) peers[r] = (r + 1 < R) ? r + 1 : -1;
        rc = oracle_sendrecv((const void *const *)send, recv, peers, n, dtype, R);
    }
    if (op == 4) rc = oracle_alltoall((const void *const *)send, recv, n, dtype, R);
    if (dtype == OR_UINT8 && op < 2) rc = rc == -2 ? 0 : 1;  /* bytes have no sum: refused */
    if (dtype == OR_BF16 && op == 0 && rc == 0)               /* bf16 partials rounded per hop */
        rc = oracle_allreduce_bf16_hops((const void *const *)send, recv, n, R);
    if (dtype == OR_BF16 && op == 1 && rc == 0)
        rc = oracle_reduce_scatter_bf16_hops((const void *const *)send, recv, n, R);
    if (rc != 0) {
        fprintf(stderr, "op %d dtype %d R %d n %zu: rc %d\n", op, dtype, R, n, rc);
        exit(1);
    }
    for (int r = 0; r < R; ++r) {
        free(send[r]);
        free(recv[r]);
    }
    ++checked;
}

static void run_v(int dtype, int R, int salt)
{
    size_t es = elem_size(dtype);
    size_t C[64 * 64], sd[64 * 64], rd[64 * 64];
    size_t smax[64] = {0}, rmax[64] = {0};
    void *send[64], *recv[64];
    for (int s = 0; s < R; ++s)
        for (int d = 0; d < R; ++d) C[s * R + d] = (size_t)((s * 5 + d * 3 + salt) % 9);
    for (int s = 0; s < R; ++s) {
        size_t off = 0;
        for (int d = 0; d < R; ++d) { sd[s * R + d] = off; off += C[s * R + d]; }
        smax[s] = off;
    }
    for (int d = 0; d < R; ++d) {
        size_t off = 0;
        for (int s = 0; s < R; ++s) { rd[s * R + d] = off; off += C[s * R + d]; }
        rmax[d] = off;
    }
    for (int r = 0; r < R; ++r) {
        send[r] = fill(smax[r] * es, dtype);
        recv[r] = fill(rmax[r] * es, dtype);
    }
    if (oracle_alltoallv((const void *const *)send, C, sd, recv, rd, dtype, R) != 0) exit(1);
    for (int r = 0; r < R; ++r) {
        free(send[r]);
        free(recv[r]);
    }
    ++checked;
}

int main(void)
{
    const int Rs[] = {1, 2, 3, 4, 5, 8, 13, 64};
    for (size_t a = 0; a < sizeof Rs / sizeof Rs[0]; ++a)
        for (int dtype = 0; dtype < 4; ++dtype) {
            int R = Rs[a];
            size_t counts[] = {0, 1, 7, (size_t)R * 5 + 3, 300};
            for (size_t k = 0; k < sizeof counts / sizeof counts[0]; ++k)
                for (int op = 0; op < 5; ++op) run_case(op, dtype, R, counts[k]);
            for (int salt = 0; salt < 3; ++salt) run_v(dtype, R, salt);
        }
    /* the exported conversion over a spread of bit patterns */
    for (uint64_t b = 0; b < (1ull << 32); b += 65537) {
        float f;
        uint32_t u = (uint32_t)b;
        memcpy(&f, &u, 4);
        (void)oracle_f32_to_bf16(f);
    }
    printf("oracle cases run: %d\n", checked);
    return 0;
}
