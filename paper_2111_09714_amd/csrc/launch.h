// Host-side launchers of the YOSO kernels (internal to libyoso).
// Arguments are assumed valid: the C ABI layer checks them first.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace yoso {

// LDS bytes that one table workgroup may use for bucket tables.
constexpr size_t kTableLdsBudget = 128 * 1024;
// Widest feature slice per table workgroup (wider slices run out of registers).
constexpr int kTableMaxDS = 16;

struct TablePlan {
    int G;        // hashes whose tables share LDS at once
    int DS;       // feature dims per workgroup
    int groups;   // ceil(m / G)
    size_t lds;   // table bytes = 2^tau * G * DS * 4
};

TablePlan plan_table(int m, int tau);
size_t table_workspace_bytes(bool bf16, int64_t bh, int64_t n_dst, int m, int tau);
size_t hash_lds_bytes(int m, int tau);

struct BackwardLayout {
    size_t qoff, koff, qent, kent, qct, kct, qs, dys, ks, vs, pq, pk, lq, lk, eq, ek, rexq, rexk, pmax, table, total;
};
BackwardLayout backward_layout(bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m, int tau);

// *YOSO: the pair layout for m*tau derived hashes of tau-1 bits, then the derived
// codes of both sides and the dV table's scratch.
struct StarLayout {
    BackwardLayout pairs;
    size_t qcodes, kcodes, table, total;
};
StarLayout backward_star_layout(bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m, int tau);

hipError_t launch_hash(const void *x, bool bf16, int64_t bh, int64_t n, const float *R, int m, int tau,
                       uint16_t *codes, hipStream_t stream);

hipError_t launch_fast_hyperplanes(const uint64_t *signs, int m, int tau, float *R, hipStream_t stream);
hipError_t launch_fast_hash(const void *x, bool bf16, int64_t bh, int64_t n, const uint64_t *signs, int m, int tau,
                            uint16_t *codes, hipStream_t stream);

hipError_t launch_table(const uint16_t *src_codes, const void *values, const uint16_t *dst_codes, void *out,
                        bool bf16, int64_t bh, int64_t n_src, int64_t n_dst, int m, int tau, void *workspace,
                        hipStream_t stream);

hipError_t launch_l2norm(const void *x, void *y, bool bf16, int64_t rows, hipStream_t stream);
hipError_t launch_l2norm_backward(const void *x, const void *dy, void *dx, bool bf16, int64_t rows,
                                  hipStream_t stream);

hipError_t launch_expect_forward(const void *q, const void *k, const void *v, void *y, bool bf16, int64_t bh,
                                 int64_t n_q, int64_t n_k, int tau, hipStream_t stream);
hipError_t launch_expect_backward(const void *q, const void *k, const void *v, const void *dy, void *dq, void *dk,
                                  void *dv, bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int tau,
                                  hipStream_t stream);

// T of the backward's rule: a bucket takes the table form when b_q b_k > T (b_q + b_k).
int backward_table_threshold();

// Short sequences over many heads (both sides at most 1024 rows): the forward as
// Y = (1/m) C V over every (query, key) pair, C counted from the codes; no workspace.
bool dense_forward_applies(int64_t bh, int64_t n_q, int64_t n_k, int m, int tau);
hipError_t launch_dense_forward(const uint16_t *qcodes, const uint16_t *kcodes, const void *v, void *y, bool bf16,
                                int64_t bh, int64_t n_q, int64_t n_k, int m, int tau, hipStream_t stream);

hipError_t launch_backward(const uint16_t *qcodes, const uint16_t *kcodes, const void *q, const void *k,
                           const void *v, const void *dy, bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m,
                           int tau, void *dq, void *dk, void *dv, void *workspace, hipStream_t stream);
hipError_t launch_backward_star(const uint16_t *qcodes, const uint16_t *kcodes, const void *q, const void *k,
                                const void *v, const void *dy, bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m,
                                int tau, void *dq, void *dk, void *dv, void *workspace, hipStream_t stream);

}  // namespace yoso
