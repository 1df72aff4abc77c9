// C ABI of libyoso: argument validation, workspace sizing and dispatch.
// Every check runs on the host before the first HIP call.
#include <stdarg.h>
#include <stdio.h>

#include <mutex>

#include "../../include/yoso.h"
#include "launch.h"

// Workspace of yoso_backward_noalloc: one copy of this array per GPU the library
// runs on, held until the process ends.  Host code never uses the name itself
// (on the host it is only a stand-in for the device symbol): it asks
// hipGetSymbolAddress for each device's address once and passes that pointer.
constexpr size_t kNoAllocScratchBytes = size_t{64} << 20;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

thread_local char g_last_error[512] = "";

yoso_status fail(yoso_status s, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return s;
}

yoso_status device_status(hipError_t e, const char *what) {
    if (e == hipSuccess) return YOSO_OK;
    return fail(YOSO_ERR_DEVICE, "%s: %s (%s)", what, hipGetErrorName(e), hipGetErrorString(e));
}

constexpr int64_t kMaxN = 65536;
constexpr int64_t kMaxGrid = 0x7fffffff;

yoso_status check_dtype(yoso_dtype dt) {
    if (dt != YOSO_F32 && dt != YOSO_BF16) return fail(YOSO_ERR_DTYPE, "unknown dtype %d", (int)dt);
    return YOSO_OK;
}

yoso_status check_shape(int64_t bh, int64_t n_q, int64_t n_k, int32_t d, int32_t m) {
    if (d != 64) return fail(YOSO_ERR_SHAPE, "d = %d; only d = 64 is supported", d);
    if (bh < 0) return fail(YOSO_ERR_SHAPE, "bh = %lld < 0", (long long)bh);
    if (n_q < 0 || n_q > kMaxN) return fail(YOSO_ERR_SHAPE, "n_q = %lld outside [0, 65536]", (long long)n_q);
    if (n_k < 0 || n_k > kMaxN) return fail(YOSO_ERR_SHAPE, "n_k = %lld outside [0, 65536]", (long long)n_k);
    // grid limits: 2*bh*m sort and pair blocks, bh*32 table blocks, bh*n/16 reduce blocks
    if (m > 0 && bh > kMaxGrid / (2 * (int64_t)m))
        return fail(YOSO_ERR_SHAPE, "bh = %lld too large for m = %d", (long long)bh, m);
    if (bh > kMaxGrid / 64) return fail(YOSO_ERR_SHAPE, "bh = %lld too large", (long long)bh);
    const int64_t nmax = n_q > n_k ? n_q : n_k;
    if (nmax > 0 && bh > kMaxGrid * 16 / nmax)
        return fail(YOSO_ERR_SHAPE, "bh*n = %lld*%lld too large", (long long)bh, (long long)nmax);
    return YOSO_OK;
}

// row operations: any number of 64-value rows (grid-stride kernels)
yoso_status check_rows(int64_t rows, int32_t d) {
    if (d != 64) return fail(YOSO_ERR_SHAPE, "d = %d; only d = 64 is supported", d);
    if (rows < 0) return fail(YOSO_ERR_SHAPE, "rows = %lld < 0", (long long)rows);
    if (rows > (int64_t{1} << 40)) return fail(YOSO_ERR_SHAPE, "rows = %lld too large", (long long)rows);
    return YOSO_OK;
}

yoso_status check_hash(int32_t m, int32_t tau) {
    if (tau < 1 || tau > 12) return fail(YOSO_ERR_TAU, "tau = %d outside [1, 12]", tau);
    if (m < 1 || m > 64) return fail(YOSO_ERR_TAU, "m = %d outside [1, 64]", m);
    if (m * tau > 512) return fail(YOSO_ERR_TAU, "m*tau = %d > 512", m * tau);
    return YOSO_OK;
}

yoso_status check_ptr(const void *p, int64_t elems, const char *name) {
    if (elems == 0) return YOSO_OK;
    if (p == nullptr) return fail(YOSO_ERR_NULL, "%s is NULL", name);
    if (reinterpret_cast<uintptr_t>(p) & 15u) return fail(YOSO_ERR_ALIGN, "%s is not 16-byte aligned", name);
    return YOSO_OK;
}

size_t required_workspace(yoso_op op, bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int32_t m, int32_t tau) {
    switch (op) {
        case YOSO_OP_HASH: return 0;
        case YOSO_OP_FORWARD:
            return yoso::dense_forward_applies(bh, n_q, n_k, m, tau) ? 0 : yoso::table_workspace_bytes(bf16, bh, n_q, m, tau);
        case YOSO_OP_BACKWARD: return yoso::backward_layout(bf16, bh, n_q, n_k, m, tau).total;
        case YOSO_OP_BACKWARD_STAR: return yoso::backward_star_layout(bf16, bh, n_q, n_k, m, tau).total;
    }
    return 0;
}

yoso_status check_workspace(const void *ws, size_t have, size_t need) {
    if (need == 0) return YOSO_OK;
    if (ws == nullptr) return fail(YOSO_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", need);
    if (have < need) return fail(YOSO_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
    if (reinterpret_cast<uintptr_t>(ws) & 15u) return fail(YOSO_ERR_ALIGN, "workspace is not 16-byte aligned");
    return YOSO_OK;
}

// The scratch array's address on the device of `stream` (which must be the
// current device), looked up on the first call on that device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices] = {};

yoso_status scratch_for(hipStream_t stream, void **ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return device_status(e, "hipGetDevice");
    if (stream != nullptr) {
        int sdev = 0;
        if ((e = hipStreamGetDevice(stream, &sdev)) != hipSuccess) return device_status(e, "hipStreamGetDevice");
        if (sdev != dev)
            return fail(YOSO_ERR_DEVICE, "the stream belongs to device %d but device %d is current", sdev, dev);
    }
    if (dev < 0 || dev >= kMaxDevices) return fail(YOSO_ERR_DEVICE, "device %d beyond the %d supported", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void *p = nullptr;
        if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess)
            return device_status(e, "hipGetSymbolAddress(scratch)");
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return YOSO_OK;
}

#define YOSO_TRY(expr)                         \
    do {                                       \
        const yoso_status _s = (expr);         \
        if (_s != YOSO_OK) return _s;          \
    } while (0)

}  // namespace

extern "C" {

const char *yoso_status_str(yoso_status status) {
    switch (status) {
        case YOSO_OK: return "ok";
        case YOSO_ERR_NULL: return "null pointer";
        case YOSO_ERR_SHAPE: return "unsupported shape";
        case YOSO_ERR_TAU: return "tau or m out of range";
        case YOSO_ERR_DTYPE: return "unknown dtype";
        case YOSO_ERR_ALIGN: return "misaligned pointer";
        case YOSO_ERR_WORKSPACE: return "workspace missing or too small";
        case YOSO_ERR_DEVICE: return "HIP error";
        case YOSO_ERR_OP: return "unknown op";
    }
    return "unknown status";
}

const char *yoso_last_error(void) { return g_last_error; }

size_t yoso_workspace_bytes(int op, int64_t bh, int64_t n_q, int64_t n_k, int32_t d, int32_t m, int32_t tau,
                            yoso_dtype dtype) {
    g_last_error[0] = '\0';
    const size_t bad = static_cast<size_t>(-1);
    if (op != YOSO_OP_HASH && op != YOSO_OP_FORWARD && op != YOSO_OP_BACKWARD && op != YOSO_OP_BACKWARD_STAR) {
        fail(YOSO_ERR_OP, "unknown op %d", op);
        return bad;
    }
    if (check_dtype(dtype) != YOSO_OK || check_shape(bh, n_q, n_k, d, m) != YOSO_OK || check_hash(m, tau) != YOSO_OK)
        return bad;
    return required_workspace(static_cast<yoso_op>(op), dtype == YOSO_BF16, bh, n_q, n_k, m, tau);
}

yoso_status yoso_hash(const void *x, yoso_dtype dtype, int64_t bh, int64_t n, int32_t d, const float *R,
                      int32_t m, int32_t tau, uint16_t *codes, void *stream) {
    g_last_error[0] = '\0';
    YOSO_TRY(check_dtype(dtype));
    YOSO_TRY(check_shape(bh, n, 0, d, m));
    YOSO_TRY(check_hash(m, tau));
    YOSO_TRY(check_ptr(x, bh * n * d, "x"));
    YOSO_TRY(check_ptr(R, (int64_t)d * m * tau, "R"));
    YOSO_TRY(check_ptr(codes, bh * n * m, "codes"));
    return device_status(yoso::launch_hash(x, dtype == YOSO_BF16, bh, n, R, m, tau, codes,
                                           static_cast<hipStream_t>(stream)),
                         "yoso_hash");
}

yoso_status yoso_fast_hyperplanes(const uint64_t *signs, int32_t d, int32_t m, int32_t tau, float *R,
                                  void *stream) {
    g_last_error[0] = '\0';
    if (d != 64) return fail(YOSO_ERR_SHAPE, "d = %d; only d = 64 is supported", d);
    YOSO_TRY(check_hash(m, tau));
    YOSO_TRY(check_ptr(signs, 3 * (((int64_t)m * tau + 63) / 64), "signs"));
    YOSO_TRY(check_ptr(R, (int64_t)d * m * tau, "R"));
    return device_status(yoso::launch_fast_hyperplanes(signs, m, tau, R, static_cast<hipStream_t>(stream)),
                         "yoso_fast_hyperplanes");
}

yoso_status yoso_fast_hash(const void *x, yoso_dtype dtype, int64_t bh, int64_t n, int32_t d,
                           const uint64_t *signs, int32_t m, int32_t tau, uint16_t *codes, void *stream) {
    g_last_error[0] = '\0';
    YOSO_TRY(check_dtype(dtype));
    YOSO_TRY(check_shape(bh, n, 0, d, m));
    YOSO_TRY(check_hash(m, tau));
    YOSO_TRY(check_ptr(x, bh * n * d, "x"));
    YOSO_TRY(check_ptr(signs, 3 * (((int64_t)m * tau + 63) / 64), "signs"));
    YOSO_TRY(check_ptr(codes, bh * n * m, "codes"));
    return device_status(yoso::launch_fast_hash(x, dtype == YOSO_BF16, bh, n, signs, m, tau, codes,
                                                static_cast<hipStream_t>(stream)),
                         "yoso_fast_hash");
}

yoso_status yoso_forward(const uint16_t *qcodes, const uint16_t *kcodes, const void *v, yoso_dtype dtype,
                         int64_t bh, int64_t n_q, int64_t n_k, int32_t d, int32_t m, int32_t tau, void *y,
                         void *workspace, size_t workspace_bytes, void *stream) {
    g_last_error[0] = '\0';
    YOSO_TRY(check_dtype(dtype));
    YOSO_TRY(check_shape(bh, n_q, n_k, d, m));
    YOSO_TRY(check_hash(m, tau));
    YOSO_TRY(check_ptr(qcodes, bh * m * n_q, "qcodes"));
    YOSO_TRY(check_ptr(kcodes, bh * m * n_k, "kcodes"));
    YOSO_TRY(check_ptr(v, bh * n_k * d, "v"));
    YOSO_TRY(check_ptr(y, bh * n_q * d, "y"));
    const bool bf16 = dtype == YOSO_BF16;
    YOSO_TRY(check_workspace(workspace, workspace_bytes, required_workspace(YOSO_OP_FORWARD, bf16, bh, n_q, n_k, m, tau)));
    if (yoso::dense_forward_applies(bh, n_q, n_k, m, tau))
        return device_status(yoso::launch_dense_forward(qcodes, kcodes, v, y, bf16, bh, n_q, n_k, m, tau,
                                                        static_cast<hipStream_t>(stream)),
                             "yoso_forward");
    return device_status(yoso::launch_table(kcodes, v, qcodes, y, bf16, bh, n_k, n_q, m, tau, workspace,
                                            static_cast<hipStream_t>(stream)),
                         "yoso_forward");
}

yoso_status yoso_backward(const uint16_t *qcodes, const uint16_t *kcodes, const void *q, const void *k,
                          const void *v, const void *dy, yoso_dtype dtype, int64_t bh, int64_t n_q, int64_t n_k,
                          int32_t d, int32_t m, int32_t tau, void *dq, void *dk, void *dv, void *workspace,
                          size_t workspace_bytes, void *stream) {
    g_last_error[0] = '\0';
    YOSO_TRY(check_dtype(dtype));
    YOSO_TRY(check_shape(bh, n_q, n_k, d, m));
    YOSO_TRY(check_hash(m, tau));
    YOSO_TRY(check_ptr(qcodes, bh * m * n_q, "qcodes"));
    YOSO_TRY(check_ptr(kcodes, bh * m * n_k, "kcodes"));
    YOSO_TRY(check_ptr(q, bh * n_q * d, "q"));
    YOSO_TRY(check_ptr(k, bh * n_k * d, "k"));
    YOSO_TRY(check_ptr(v, bh * n_k * d, "v"));
    YOSO_TRY(check_ptr(dy, bh * n_q * d, "dy"));
    YOSO_TRY(check_ptr(dq, bh * n_q * d, "dq"));
    YOSO_TRY(check_ptr(dk, bh * n_k * d, "dk"));
    YOSO_TRY(check_ptr(dv, bh * n_k * d, "dv"));
    const bool bf16 = dtype == YOSO_BF16;
    YOSO_TRY(check_workspace(workspace, workspace_bytes, required_workspace(YOSO_OP_BACKWARD, bf16, bh, n_q, n_k, m, tau)));
    return device_status(yoso::launch_backward(qcodes, kcodes, q, k, v, dy, bf16, bh, n_q, n_k, m, tau, dq, dk, dv,
                                               workspace, static_cast<hipStream_t>(stream)),
                         "yoso_backward");
}

yoso_status yoso_backward_star(const uint16_t *qcodes, const uint16_t *kcodes, const void *q, const void *k,
                               const void *v, const void *dy, yoso_dtype dtype, int64_t bh, int64_t n_q, int64_t n_k,
                               int32_t d, int32_t m, int32_t tau, void *dq, void *dk, void *dv, void *workspace,
                               size_t workspace_bytes, void *stream) {
    g_last_error[0] = '\0';
    YOSO_TRY(check_dtype(dtype));
    YOSO_TRY(check_shape(bh, n_q, n_k, d, m * tau));
    YOSO_TRY(check_hash(m, tau));
    YOSO_TRY(check_ptr(qcodes, bh * m * n_q, "qcodes"));
    YOSO_TRY(check_ptr(kcodes, bh * m * n_k, "kcodes"));
    YOSO_TRY(check_ptr(q, bh * n_q * d, "q"));
    YOSO_TRY(check_ptr(k, bh * n_k * d, "k"));
    YOSO_TRY(check_ptr(v, bh * n_k * d, "v"));
    YOSO_TRY(check_ptr(dy, bh * n_q * d, "dy"));
    YOSO_TRY(check_ptr(dq, bh * n_q * d, "dq"));
    YOSO_TRY(check_ptr(dk, bh * n_k * d, "dk"));
    YOSO_TRY(check_ptr(dv, bh * n_k * d, "dv"));
    const bool bf16 = dtype == YOSO_BF16;
    YOSO_TRY(check_workspace(workspace, workspace_bytes,
                             required_workspace(YOSO_OP_BACKWARD_STAR, bf16, bh, n_q, n_k, m, tau)));
    return device_status(yoso::launch_backward_star(qcodes, kcodes, q, k, v, dy, bf16, bh, n_q, n_k, m, tau, dq, dk,
                                                    dv, workspace, static_cast<hipStream_t>(stream)),
                         "yoso_backward_star");
}

yoso_status yoso_backward_noalloc(const uint16_t *qcodes, const uint16_t *kcodes, const void *q, const void *k,
                                  const void *v, const void *dy, yoso_dtype dtype, int64_t bh, int64_t n_q,
                                  int64_t n_k, int32_t d, int32_t m, int32_t tau, void *dq, void *dk, void *dv,
                                  void *stream) {
    g_last_error[0] = '\0';
    YOSO_TRY(check_dtype(dtype));
    YOSO_TRY(check_shape(bh, n_q, n_k, d, m));
    YOSO_TRY(check_hash(m, tau));
    YOSO_TRY(check_ptr(qcodes, bh * m * n_q, "qcodes"));
    YOSO_TRY(check_ptr(kcodes, bh * m * n_k, "kcodes"));
    YOSO_TRY(check_ptr(q, bh * n_q * d, "q"));
    YOSO_TRY(check_ptr(k, bh * n_k * d, "k"));
    YOSO_TRY(check_ptr(v, bh * n_k * d, "v"));
    YOSO_TRY(check_ptr(dy, bh * n_q * d, "dy"));
    YOSO_TRY(check_ptr(dq, bh * n_q * d, "dq"));
    YOSO_TRY(check_ptr(dk, bh * n_k * d, "dk"));
    YOSO_TRY(check_ptr(dv, bh * n_k * d, "dv"));
    const bool bf16 = dtype == YOSO_BF16;
    const size_t need = required_workspace(YOSO_OP_BACKWARD, bf16, bh, n_q, n_k, m, tau);
    if (need > kNoAllocScratchBytes)
        return fail(YOSO_ERR_WORKSPACE,
                    "these shapes need %zu bytes of scratch; yoso_backward_noalloc has %zu (use yoso_backward with a "
                    "workspace)",
                    need, kNoAllocScratchBytes);
    const hipStream_t s = static_cast<hipStream_t>(stream);
    void *ws = nullptr;
    if (need > 0) YOSO_TRY(scratch_for(s, &ws));
    return device_status(yoso::launch_backward(qcodes, kcodes, q, k, v, dy, bf16, bh, n_q, n_k, m, tau, dq, dk, dv,
                                               ws, s),
                         "yoso_backward_noalloc");
}

size_t yoso_backward_noalloc_limit(void) { return kNoAllocScratchBytes; }

int32_t yoso_backward_table_threshold(void) { return yoso::backward_table_threshold(); }

yoso_status yoso_l2_normalize(const void *x, yoso_dtype dtype, int64_t rows, int32_t d, void *y, void *stream) {
    g_last_error[0] = '\0';
    YOSO_TRY(check_dtype(dtype));
    YOSO_TRY(check_rows(rows, d));
    YOSO_TRY(check_ptr(x, rows * d, "x"));
    YOSO_TRY(check_ptr(y, rows * d, "y"));
    return device_status(yoso::launch_l2norm(x, y, dtype == YOSO_BF16, rows, static_cast<hipStream_t>(stream)),
                         "yoso_l2_normalize");
}

yoso_status yoso_l2_normalize_backward(const void *x, const void *dy, yoso_dtype dtype, int64_t rows, int32_t d,
                                       void *dx, void *stream) {
    g_last_error[0] = '\0';
    YOSO_TRY(check_dtype(dtype));
    YOSO_TRY(check_rows(rows, d));
    YOSO_TRY(check_ptr(x, rows * d, "x"));
    YOSO_TRY(check_ptr(dy, rows * d, "dy"));
    YOSO_TRY(check_ptr(dx, rows * d, "dx"));
    return device_status(
        yoso::launch_l2norm_backward(x, dy, dx, dtype == YOSO_BF16, rows, static_cast<hipStream_t>(stream)),
        "yoso_l2_normalize_backward");
}

yoso_status yoso_expectation_forward(const void *q, const void *k, const void *v, yoso_dtype dtype, int64_t bh,
                                     int64_t n_q, int64_t n_k, int32_t d, int32_t tau, void *y, void *stream) {
    g_last_error[0] = '\0';
    YOSO_TRY(check_dtype(dtype));
    YOSO_TRY(check_shape(bh, n_q, n_k, d, 1));
    YOSO_TRY(check_hash(1, tau));
    YOSO_TRY(check_ptr(q, bh * n_q * d, "q"));
    YOSO_TRY(check_ptr(k, bh * n_k * d, "k"));
    YOSO_TRY(check_ptr(v, bh * n_k * d, "v"));
    YOSO_TRY(check_ptr(y, bh * n_q * d, "y"));
    return device_status(yoso::launch_expect_forward(q, k, v, y, dtype == YOSO_BF16, bh, n_q, n_k, tau,
                                                     static_cast<hipStream_t>(stream)),
                         "yoso_expectation_forward");
}

yoso_status yoso_expectation_backward(const void *q, const void *k, const void *v, const void *dy, yoso_dtype dtype,
                                      int64_t bh, int64_t n_q, int64_t n_k, int32_t d, int32_t tau, void *dq,
                                      void *dk, void *dv, void *stream) {
    g_last_error[0] = '\0';
    YOSO_TRY(check_dtype(dtype));
    YOSO_TRY(check_shape(bh, n_q, n_k, d, 1));
    YOSO_TRY(check_hash(1, tau));
    YOSO_TRY(check_ptr(q, bh * n_q * d, "q"));
    YOSO_TRY(check_ptr(k, bh * n_k * d, "k"));
    YOSO_TRY(check_ptr(v, bh * n_k * d, "v"));
    YOSO_TRY(check_ptr(dy, bh * n_q * d, "dy"));
    YOSO_TRY(check_ptr(dq, bh * n_q * d, "dq"));
    YOSO_TRY(check_ptr(dk, bh * n_k * d, "dk"));
    YOSO_TRY(check_ptr(dv, bh * n_k * d, "dv"));
    return device_status(yoso::launch_expect_backward(q, k, v, dy, dq, dk, dv, dtype == YOSO_BF16, bh, n_q, n_k, tau,
                                                      static_cast<hipStream_t>(stream)),
                         "yoso_expectation_backward");
}

}  // extern "C"
