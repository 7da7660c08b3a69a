/* The C ABI used from plain C, with no Python and no torch: buffers from
 * hipMalloc, every collective once on a stream of its own, results read
 * back and checked against closed forms (int32 sums of x_r[i] = r*K + i,
 * which wrap-around arithmetic makes independent of the summation order) and
 * bit-for-bit copies; then the documented argument errors.  Exit status 0
 * and the line "c abi ok" mean every check passed. */
#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../include/hoccl.h"

/* Sizes the Python binding mirrors (tests/test_abi.py checks the same). */
#define HOCCL_CONFIG_SIZE 96
#define HOCCL_STATS_SIZE 56

#define R 5
#define N 1003 /* ragged against R */

/* The boundary's enum values and struct layouts, pinned at compile time:
 * the copy paths keep AUTO 0, SDMA 1, KERNEL 2 (HIP appended as 3), and
 * the configuration and statistics keep their core fields first, in order,
 * with the extensions after them. */
_Static_assert(HOCCL_OK == 0 && HOCCL_ERR_INVALID_ARG == 1 && HOCCL_ERR_UNSUPPORTED == 2 &&
               HOCCL_ERR_HIP == 3 && HOCCL_ERR_NO_MEMORY == 4 && HOCCL_ERR_TIMEOUT == 5 &&
               HOCCL_ERR_INTERNAL == 6, "status values");
_Static_assert(HOCCL_INT32 == 0 && HOCCL_FP32 == 1 && HOCCL_BF16 == 2 && HOCCL_UINT8 == 3,
               "dtype values");
_Static_assert(HOCCL_COPY_AUTO == 0 && HOCCL_COPY_SDMA == 1 && HOCCL_COPY_KERNEL == 2 &&
               HOCCL_COPY_HIP == 3, "copy path values");
_Static_assert(HOCCL_REDUCE_RING == 0 && HOCCL_REDUCE_DIRECT == 1 && HOCCL_REDUCE_AUTO == 2,
               "reduction algorithm values");
_Static_assert(offsetof(hoccl_config_t, workgroups_per_step) == 0 &&
               offsetof(hoccl_config_t, threads_per_workgroup) == 4 &&
               offsetof(hoccl_config_t, chunk_bytes) == 8 &&
               offsetof(hoccl_config_t, copy_streams) == 16 &&
               offsetof(hoccl_config_t, copy_path) == 20 &&
               offsetof(hoccl_config_t, allgather_direct) == 24 &&
               offsetof(hoccl_config_t, allreduce_chunk_groups) == 28, "core configuration layout");
_Static_assert(offsetof(hoccl_stats_t, reduce_launches) == 0 && offsetof(hoccl_stats_t, copy_ops) == 4 &&
               offsetof(hoccl_stats_t, workgroups_per_step) == 8 &&
               offsetof(hoccl_stats_t, cus_available) == 12 &&
               offsetof(hoccl_stats_t, cus_used_max) == 16 &&
               offsetof(hoccl_stats_t, copy_path_used) == 20 &&
               offsetof(hoccl_stats_t, hbm_bytes_algorithmic) == 24 &&
               offsetof(hoccl_stats_t, host_enqueue_us) == 32, "core statistics layout");
_Static_assert(sizeof(hoccl_config_t) == HOCCL_CONFIG_SIZE, "configuration size");
_Static_assert(sizeof(hoccl_stats_t) == HOCCL_STATS_SIZE, "statistics size");

static int failures = 0;
#define CHECK(cond, ...)                                  \
    do {                                                  \
        if (!(cond)) {                                    \
            fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
            fprintf(stderr, __VA_ARGS__);                 \
            fprintf(stderr, "\n");                        \
            ++failures;                                   \
        }                                                 \
    } while (0)
#define HIP_OK(call)                                                          \
    do {                                                                      \
        hipError_t e_ = (call);                                               \
        if (e_ != hipSuccess) {                                               \
            fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));        \
            exit(2);                                                          \
        }                                                                     \
    } while (0)
#define HOCCL_OK_(call)                                                       \
    do {                                                                      \
        hoccl_status_t s_ = (call);                                           \
        if (s_ != HOCCL_OK) {                                                 \
            fprintf(stderr, "%s: %s (%s)\n", #call, hoccl_status_string(s_),  \
                    hoccl_last_error_string());                               \
            exit(3);                                                          \
        }                                                                     \
    } while (0)

static int32_t *dev_alloc(size_t n) {
    void *p = NULL;
    HIP_OK(hipMalloc(&p, n * sizeof(int32_t) + 16));
    return (int32_t *)p;
}

int main(void) {
    HIP_OK(hipSetDevice(0));
    HOCCL_OK_(hoccl_init(0));
    hipStream_t s;
    HIP_OK(hipStreamCreate(&s));
    const uint32_t K = 1u << 28; /* r*K + i wraps for r >= 8 in int32 sums */
    int32_t *send[R], *recv[R];
    int32_t *h = malloc(sizeof(int32_t) * R * (size_t)N * R);
    int32_t *g = malloc(sizeof(int32_t) * R * (size_t)N * R);

    /* reduce-scatter, int32: recv_r[i] = sum_s x_s[r*N + i] */
    for (int r = 0; r < R; ++r) {
        send[r] = dev_alloc((size_t)R * N);
        recv[r] = dev_alloc((size_t)R * N);
        for (size_t i = 0; i < (size_t)R * N; ++i) h[i] = (int32_t)((uint32_t)r * K + (uint32_t)i);
        HIP_OK(hipMemcpy(send[r], h, sizeof(int32_t) * R * N, hipMemcpyHostToDevice));
    }
    HOCCL_OK_(hoccl_reduce_scatter((const void *const *)send, (void *const *)recv, N, HOCCL_INT32, R, s));
    HIP_OK(hipStreamSynchronize(s));
    for (int r = 0; r < R; ++r) {
        HIP_OK(hipMemcpy(g, recv[r], sizeof(int32_t) * N, hipMemcpyDeviceToHost));
        for (size_t i = 0; i < N; ++i) {
            uint32_t want = 0;
            for (int q = 0; q < R; ++q) want += (uint32_t)q * K + (uint32_t)(r * N + i);
            CHECK((uint32_t)g[i] == want, "reduce-scatter rank %d elem %zu", r, i);
        }
    }
    hoccl_stats_t st;
    HOCCL_OK_(hoccl_get_last_stats(&st));
    CHECK(st.reduce_launches >= 1 && st.hbm_bytes_algorithmic > 0, "stats after reduce-scatter");

    /* all-reduce, int32, in place: every element is the sum over ranks */
    HOCCL_OK_(hoccl_allreduce((const void *const *)send, (void *const *)send, (size_t)R * N, HOCCL_INT32, R, s));
    HIP_OK(hipStreamSynchronize(s));
    for (int r = 0; r < R; ++r) {
        HIP_OK(hipMemcpy(g, send[r], sizeof(int32_t) * R * N, hipMemcpyDeviceToHost));
        for (size_t i = 0; i < (size_t)R * N; ++i) {
            uint32_t want = 0;
            for (int q = 0; q < R; ++q) want += (uint32_t)q * K + (uint32_t)i;
            CHECK((uint32_t)g[i] == want, "all-reduce rank %d elem %zu", r, i);
        }
    }

    /* all-gather: recv_r[q*N + i] = x_q[i], bitwise, on each copy path */
    for (int path = HOCCL_COPY_AUTO; path <= HOCCL_COPY_HIP; ++path) {
        hoccl_config_t cfg;
        HOCCL_OK_(hoccl_get_config(&cfg));
        cfg.copy_path = (hoccl_copy_path_t)path;
        HOCCL_OK_(hoccl_set_config(&cfg));
        for (int r = 0; r < R; ++r) {
            for (size_t i = 0; i < N; ++i) h[i] = (int32_t)(0x9e3779b9u * (uint32_t)(r * N + i + path));
            HIP_OK(hipMemcpy(send[r], h, sizeof(int32_t) * N, hipMemcpyHostToDevice));
        }
        hoccl_status_t st2 = hoccl_allgather((const void *const *)send, (void *const *)recv, N, HOCCL_INT32, R, s);
        if (path == HOCCL_COPY_SDMA && st2 == HOCCL_ERR_UNSUPPORTED) continue;
        HOCCL_OK_(st2);
        HIP_OK(hipStreamSynchronize(s));
        for (int r = 0; r < R; ++r) {
            HIP_OK(hipMemcpy(g, recv[r], sizeof(int32_t) * R * N, hipMemcpyDeviceToHost));
            for (int q = 0; q < R; ++q)
                for (size_t i = 0; i < N; ++i)
                    CHECK((uint32_t)g[(size_t)q * N + i] == 0x9e3779b9u * (uint32_t)(q * N + i + path),
                          "all-gather path %d rank %d block %d elem %zu", path, r, q, i);
        }
    }
    hoccl_config_t cfg;
    HOCCL_OK_(hoccl_get_config(&cfg));
    cfg.copy_path = HOCCL_COPY_AUTO;
    HOCCL_OK_(hoccl_set_config(&cfg));

    /* all-to-all: recv_d[q*N + i] = x_q[d*N + i] */
    for (int r = 0; r < R; ++r) {
        for (size_t i = 0; i < (size_t)R * N; ++i) h[i] = (int32_t)(r * 1000003 + i);
        HIP_OK(hipMemcpy(send[r], h, sizeof(int32_t) * R * N, hipMemcpyHostToDevice));
    }
    HOCCL_OK_(hoccl_alltoall((const void *const *)send, (void *const *)recv, N, HOCCL_INT32, R, s));
    HIP_OK(hipStreamSynchronize(s));
    for (int d = 0; d < R; ++d) {
        HIP_OK(hipMemcpy(g, recv[d], sizeof(int32_t) * R * N, hipMemcpyDeviceToHost));
        for (int q = 0; q < R; ++q)
            for (size_t i = 0; i < N; ++i)
                CHECK(g[(size_t)q * N + i] == (int32_t)(q * 1000003 + d * N + i), "all-to-all %d %d", d, q);
    }

    /* send/recv r -> r+1, the last rank sends nothing: recv_0 untouched */
    HIP_OK(hipMemset(recv[0], 0x5a, sizeof(int32_t) * N));
    int peers[R];
    for (int r = 0; r < R; ++r) peers[r] = r + 1 < R ? r + 1 : -1;
    HOCCL_OK_(hoccl_sendrecv((const void *const *)send, (void *const *)recv, peers, N, HOCCL_INT32, R, s));
    HIP_OK(hipStreamSynchronize(s));
    HIP_OK(hipMemcpy(g, recv[0], sizeof(int32_t) * N, hipMemcpyDeviceToHost));
    for (size_t i = 0; i < N; ++i) CHECK(g[i] == 0x5a5a5a5a, "send/recv touched a non-receiver");
    for (int d = 1; d < R; ++d) {
        HIP_OK(hipMemcpy(g, recv[d], sizeof(int32_t) * N, hipMemcpyDeviceToHost));
        for (size_t i = 0; i < N; ++i) CHECK(g[i] == (int32_t)((d - 1) * 1000003 + i), "send/recv %d", d);
    }

    /* one ring hop, int32 (wrapping): out[i] = a[i] + b[i] mod 2^32, written
     * in place over a */
    for (size_t i = 0; i < N; ++i) h[i] = (int32_t)(0x7ffffff0u + (uint32_t)i);
    HIP_OK(hipMemcpy(send[0], h, sizeof(int32_t) * N, hipMemcpyHostToDevice));
    for (size_t i = 0; i < N; ++i) h[i] = (int32_t)(3u * (uint32_t)i + 1u);
    HIP_OK(hipMemcpy(send[1], h, sizeof(int32_t) * N, hipMemcpyHostToDevice));
    HOCCL_OK_(hoccl_ring_hop(send[0], send[1], send[0], N, HOCCL_INT32, HOCCL_HOP_MIDDLE, s));
    HIP_OK(hipStreamSynchronize(s));
    HIP_OK(hipMemcpy(g, send[0], sizeof(int32_t) * N, hipMemcpyDeviceToHost));
    for (size_t i = 0; i < N; ++i)
        CHECK(g[i] == (int32_t)(0x7ffffff0u + (uint32_t)i + 3u * (uint32_t)i + 1u), "ring hop %zu", i);
    CHECK(hoccl_ring_hop(send[0], send[1], send[0], N, HOCCL_INT32, (hoccl_hop_t)7, s) ==
              HOCCL_ERR_INVALID_ARG, "unknown hop accepted");

    /* documented argument errors enqueue nothing and say why */
    CHECK(hoccl_allreduce((const void *const *)send, (void *const *)recv, N, HOCCL_INT32, 0, s) ==
              HOCCL_ERR_INVALID_ARG, "R = 0 accepted");
    CHECK(hoccl_allreduce(NULL, (void *const *)recv, N, HOCCL_INT32, R, s) == HOCCL_ERR_INVALID_ARG,
          "null send array accepted");
    int dup[R];
    for (int r = 0; r < R; ++r) dup[r] = 1;
    CHECK(hoccl_sendrecv((const void *const *)send, (void *const *)recv, dup, N, HOCCL_INT32, R, s) ==
              HOCCL_ERR_INVALID_ARG, "duplicate receiver accepted");
    CHECK(strlen(hoccl_last_error_string()) > 0, "no error text");
    CHECK(hoccl_allreduce((const void *const *)send, (void *const *)recv, 0, HOCCL_INT32, R, s) == HOCCL_OK,
          "count 0 is not a no-op");

    HIP_OK(hipStreamSynchronize(s));
    for (int r = 0; r < R; ++r) {
        HIP_OK(hipFree(send[r]));
        HIP_OK(hipFree(recv[r]));
    }
    HIP_OK(hipStreamDestroy(s));
    HOCCL_OK_(hoccl_finalize());
    free(h);
    free(g);
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("c abi ok\n");
    return 0;
}
