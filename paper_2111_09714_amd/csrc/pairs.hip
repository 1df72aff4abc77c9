// Backward dQ, dK of YOSO attention on MFMA (gfx950).
//
// Sec. 3.3, eq. (pseudo-gradient-q) evaluated on the sampled collisions:
//   dQ = tau/(2m) sum_h [(dY V^T) .* B_h] K,   dK = tau/(2m) sum_h [(dY V^T) .* B_h]^T Q.
// For one hash the nonzeros of B_h form blocks: query bucket c meets key
// bucket c.  Sorting the rows of Q and K by code turns B_h into a block-diagonal
// matrix in (sorted query, sorted key) coordinates.  This is the same sum the
// paper writes as d runs of the table subroutine (eq. backward-d2), evaluated
// pair by pair (3d multiply-adds per colliding pair instead of 2d^2 per row).
//
// Kernels:
//   sort_kernel   one workgroup per (head, hash, side): histogram of the codes,
//                 exclusive scan -> bucket offsets, then row ids and codes in
//                 bucket order (a counting sort in LDS).
//   pairs_kernel  one workgroup per (head, hash).  Each wave walks 16-row tiles
//                 of sorted queries; the keys that can collide with a tile form
//                 one contiguous range of sorted keys, visited 16 at a time:
//                   S^T = V_k dY_q^T and S = dY_q V_k^T   (16x16x32 MFMA, 2 k-steps)
//                   mask by code equality, scale by tau/(2m)
//                   dQ^T_q += K_k^T S^T,  dK^T_k = Q_q^T S  (16x16x16 MFMA)
//                 The MFMA output layout of S^T / S is directly the B operand of
//                 the 16x16x16 products, so no register shuffles are needed.
//                 dQ of a tile is accumulated over its key range and added once;
//                 dK of each key tile is added per query tile.  Both go into fp32
//                 buffers with global atomics (the m hashes of a row land in
//                 different workgroups).
// Every fp32 product uses three fp16 MFMAs (hi*hi + hi*lo + lo*hi); Q and K are
// scaled by 2^8 before splitting (undone on the way out).
#include "common.h"
#include "launch.h"
#include "timing.h"

namespace yoso {

namespace {

constexpr int kSortThreads = 256;
constexpr int kPairThreads = 256;

// ---------------------------------------------------------------- counting sort
__global__ __launch_bounds__(kSortThreads) void sort_kernel(const uint16_t *__restrict__ qcodes,
                                                            const uint16_t *__restrict__ kcodes, int64_t units,
                                                            int64_t n_q, int64_t n_k, int tau,
                                                            int32_t *__restrict__ qoff, int32_t *__restrict__ koff,
                                                            uint16_t *__restrict__ qperm,
                                                            uint16_t *__restrict__ kperm,
                                                            uint16_t *__restrict__ qsorted,
                                                            uint16_t *__restrict__ ksorted) {
    extern __shared__ int32_t cnt[];  // [buckets] counts, then cursors; + [kSortThreads] scan scratch
    int32_t *scan = cnt + (1 << tau);
    const int64_t unit = blockIdx.x >> 1;
    const bool kside = blockIdx.x & 1;
    const int64_t n = kside ? n_k : n_q;
    const uint16_t *codes = (kside ? kcodes : qcodes) + unit * n;
    int32_t *off = (kside ? koff : qoff) + unit * ((1 << tau) + 1);
    uint16_t *perm = (kside ? kperm : qperm) + unit * n;
    uint16_t *sorted = (kside ? ksorted : qsorted) + unit * n;
    const int B = 1 << tau;
    const int tid = threadIdx.x;

    for (int c = tid; c < B; c += kSortThreads) cnt[c] = 0;
    __syncthreads();
    for (int64_t i = tid; i < n; i += kSortThreads) atomicAdd(&cnt[codes[i] & (B - 1)], 1);
    __syncthreads();

    // exclusive scan: thread t owns buckets [t*per, (t+1)*per)
    const int per = (B + kSortThreads - 1) / kSortThreads;
    const int c0 = tid * per;
    int32_t local = 0;
    for (int c = c0; c < c0 + per && c < B; c++) local += cnt[c];
    scan[tid] = local;
    __syncthreads();
    for (int s = 1; s < kSortThreads; s <<= 1) {
        const int32_t v = (tid >= s) ? scan[tid - s] : 0;
        __syncthreads();
        scan[tid] += v;
        __syncthreads();
    }
    int32_t run = scan[tid] - local;  // exclusive prefix of this thread's first bucket
    for (int c = c0; c < c0 + per && c < B; c++) {
        const int32_t k = cnt[c];
        off[c] = run;
        cnt[c] = run;  // becomes the cursor
        run += k;
    }
    if (tid == 0) off[B] = static_cast<int32_t>(n);
    __syncthreads();

    for (int64_t i = tid; i < n; i += kSortThreads) {
        const int c = codes[i] & (B - 1);
        const int32_t pos = atomicAdd(&cnt[c], 1);
        perm[pos] = static_cast<uint16_t>(i);
        sorted[pos] = static_cast<uint16_t>(c);
    }
}

// ---------------------------------------------------------------- pairs
struct PairArgs {
    const void *q, *k, *v, *dy;          // [bh][n][64]
    const int32_t *qoff, *koff;          // [units][2^tau + 1]
    const uint16_t *qperm, *kperm;       // [units][n]
    const uint16_t *qsorted, *ksorted;   // [units][n]
    float *dq, *dk;                      // fp32 accumulators [bh][n][64]
    int64_t bh, n_q, n_k;
    int m, tau;
    float scale;                         // tau / (2m)
};

template <bool BF16>
__global__ __launch_bounds__(kPairThreads) void pairs_kernel(PairArgs a) {
    const int64_t units = a.bh * a.m;
    const int64_t unit = xcd_remap(blockIdx.x, units);
    const int64_t b = unit / a.m;
    const int nb = (1 << a.tau) + 1;
    const int32_t *koff = a.koff + unit * nb;
    const uint16_t *qperm = a.qperm + unit * a.n_q;
    const uint16_t *kperm = a.kperm + unit * a.n_k;
    const uint16_t *qsorted = a.qsorted + unit * a.n_q;
    const uint16_t *ksorted = a.ksorted + unit * a.n_k;
    const int64_t qrow0 = b * a.n_q, krow0 = b * a.n_k;

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, c = lane & 15;
    const int64_t qtiles = (a.n_q + 15) >> 4;

    for (int64_t qt = wave; qt < qtiles; qt += kPairThreads / 64) {
        const int64_t p0 = qt * 16;
        const int64_t plast = (p0 + 15 < a.n_q) ? p0 + 15 : a.n_q - 1;
        const int cfirst = qsorted[p0], clast = qsorted[plast];
        const int64_t kbeg = koff[cfirst], kend = koff[clast + 1];
        if (kbeg >= kend) continue;

        // ---- query-side operands
        // dY rows as 16x16x32 fragments: lane (g, c) holds row p0+c, dims kb*32 + g*8 + [0,8)
        const bool qv_c = p0 + c < a.n_q;
        const int64_t qrow_c = qv_c ? qrow0 + qperm[p0 + c] : 0;
        half8 dyh[2], dyl[2];
#pragma unroll
        for (int kb = 0; kb < 2; kb++) {
            float t[8];
            if (qv_c) {
                load8<BF16>(a.dy, qrow_c * D + kb * 32 + g * 8, t);
            } else {
#pragma unroll
                for (int i = 0; i < 8; i++) t[i] = 0.f;
            }
            split8(t, 1.0f, dyh[kb], dyl[kb]);
        }
        // Q^T as 16x16x16 A fragments: lane (g, c) holds dims 16dt + c of rows p0 + 4g + [0,4)
        int qcode_r[4];
        int64_t qrow_r[4];
        bool qv_r[4];
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const int64_t p = p0 + 4 * g + i;
            qv_r[i] = p < a.n_q;
            qrow_r[i] = qv_r[i] ? qrow0 + qperm[p] : 0;
            qcode_r[i] = qv_r[i] ? qsorted[p] : -1;
        }
        half4 qh[4], ql[4];
#pragma unroll
        for (int dt = 0; dt < 4; dt++) {
            float t[4];
#pragma unroll
            for (int i = 0; i < 4; i++) t[i] = qv_r[i] ? load1<BF16>(a.q, qrow_r[i] * D + dt * 16 + c) : 0.f;
            split4(t, 256.0f, qh[dt], ql[dt]);
        }
        const int qcode_c = qv_c ? qsorted[p0 + c] : -2;

        floatx4 dqT[4];
#pragma unroll
        for (int dt = 0; dt < 4; dt++) dqT[dt] = floatx4{0.f, 0.f, 0.f, 0.f};

        for (int64_t k0 = kbeg; k0 < kend; k0 += 16) {
            // ---- key-side operands
            const bool kv_c = k0 + c < kend;
            const int64_t krow_c = kv_c ? krow0 + kperm[k0 + c] : 0;
            half8 vh[2], vl[2];
#pragma unroll
            for (int kb = 0; kb < 2; kb++) {
                float t[8];
                if (kv_c) {
                    load8<BF16>(a.v, krow_c * D + kb * 32 + g * 8, t);
                } else {
#pragma unroll
                    for (int i = 0; i < 8; i++) t[i] = 0.f;
                }
                split8(t, 1.0f, vh[kb], vl[kb]);
            }
            int kcode_r[4];
            int64_t krow_r[4];
            bool kv_r[4];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int64_t p = k0 + 4 * g + i;
                kv_r[i] = p < kend;
                krow_r[i] = kv_r[i] ? krow0 + kperm[p] : 0;
                kcode_r[i] = kv_r[i] ? ksorted[p] : -3;
            }
            half4 kh[4], kl[4];
#pragma unroll
            for (int dt = 0; dt < 4; dt++) {
                float t[4];
#pragma unroll
                for (int i = 0; i < 4; i++)
                    t[i] = kv_r[i] ? load1<BF16>(a.k, krow_r[i] * D + dt * 16 + c) : 0.f;
                split4(t, 256.0f, kh[dt], kl[dt]);
            }
            const int kcode_c = kv_c ? ksorted[k0 + c] : -4;

            // ---- S^T[key 4g+i][query c] and S[query 4g+i][key c]
            floatx4 st = {0.f, 0.f, 0.f, 0.f}, s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kb = 0; kb < 2; kb++) {
                st = mfma3_16x16x32(vh[kb], vl[kb], dyh[kb], dyl[kb], st);
                s = mfma3_16x16x32(dyh[kb], dyl[kb], vh[kb], vl[kb], s);
            }
            float stv[4], sv[4];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                stv[i] = (kcode_r[i] == qcode_c) ? st[i] * a.scale : 0.f;
                sv[i] = (qcode_r[i] == kcode_c) ? s[i] * a.scale : 0.f;
            }
            half4 sth, stl, sh, sl;
            split4(stv, 1.0f, sth, stl);
            split4(sv, 1.0f, sh, sl);

            // ---- dQ^T += K^T S^T ; dK^T = Q^T S
            floatx4 dkT[4];
#pragma unroll
            for (int dt = 0; dt < 4; dt++) {
                dqT[dt] = mfma3_16x16x16(kh[dt], kl[dt], sth, stl, dqT[dt]);
                dkT[dt] = mfma3_16x16x16(qh[dt], ql[dt], sh, sl, floatx4{0.f, 0.f, 0.f, 0.f});
            }
            // lane (g, c) holds dK^T[dim 16dt + 4g + i][key c]
            if (kv_c) {
                float *dst = a.dk + krow_c * D + 4 * g;
#pragma unroll
                for (int dt = 0; dt < 4; dt++)
#pragma unroll
                    for (int i = 0; i < 4; i++) unsafeAtomicAdd(dst + dt * 16 + i, dkT[dt][i] * (1.0f / 256.0f));
            }
        }
        // lane (g, c) holds dQ^T[dim 16dt + 4g + i][query c]
        if (qv_c) {
            float *dst = a.dq + qrow_c * D + 4 * g;
#pragma unroll
            for (int dt = 0; dt < 4; dt++)
#pragma unroll
                for (int i = 0; i < 4; i++) unsafeAtomicAdd(dst + dt * 16 + i, dqT[dt][i] * (1.0f / 256.0f));
        }
    }
}

__global__ void zero_kernel(float *__restrict__ p, int64_t count) {
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x)
        p[e] = 0.f;
}

__global__ void to_bf16_kernel(const float *__restrict__ in, uint16_t *__restrict__ out, int64_t count) {
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x)
        out[e] = f32_to_bf16(in[e]);
}

unsigned elementwise_grid(int64_t count) {
    const int64_t blocks = (count + 255) / 256;
    return (unsigned)(blocks < 8192 ? (blocks > 0 ? blocks : 1) : 8192);
}

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

BackwardLayout backward_layout(bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m, int tau) {
    BackwardLayout L;
    const int64_t units = bh * m;
    const size_t nb = ((size_t)1 << tau) + 1;
    size_t o = 0;
    L.qoff = o; o = align_up(o + units * nb * 4);
    L.koff = o; o = align_up(o + units * nb * 4);
    L.qperm = o; o = align_up(o + units * n_q * 2);
    L.kperm = o; o = align_up(o + units * n_k * 2);
    L.qsorted = o; o = align_up(o + units * n_q * 2);
    L.ksorted = o; o = align_up(o + units * n_k * 2);
    if (bf16) {
        L.dq_acc = o; o = align_up(o + bh * n_q * D * 4);
        L.dk_acc = o; o = align_up(o + bh * n_k * D * 4);
    } else {
        L.dq_acc = L.dk_acc = (size_t)-1;
    }
    L.table = o; o = align_up(o + table_workspace_bytes(bf16, bh, n_k, m, tau));
    L.total = o;
    return L;
}

hipError_t launch_backward(const uint16_t *qcodes, const uint16_t *kcodes, const void *q, const void *k,
                           const void *v, const void *dy, bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m,
                           int tau, void *dq, void *dk, void *dv, void *workspace, hipStream_t stream) {
    hipError_t e;
    const BackwardLayout L = backward_layout(bf16, bh, n_q, n_k, m, tau);
    unsigned char *ws = static_cast<unsigned char *>(workspace);

    // dV: the forward's table machinery with the roles of queries and keys swapped.
    e = launch_table(qcodes, dy, kcodes, dv, bf16, bh, n_q, n_k, m, tau, ws + L.table, stream);
    if (e != hipSuccess) return e;

    float *dq32 = bf16 ? reinterpret_cast<float *>(ws + L.dq_acc) : static_cast<float *>(dq);
    float *dk32 = bf16 ? reinterpret_cast<float *>(ws + L.dk_acc) : static_cast<float *>(dk);
    const int64_t nq_el = bh * n_q * D, nk_el = bh * n_k * D;
    {
        KernelTimer timer("zero_kernel", stream);
        if (nq_el) hipLaunchKernelGGL(zero_kernel, dim3(elementwise_grid(nq_el)), dim3(256), 0, stream, dq32, nq_el);
        if (nk_el) hipLaunchKernelGGL(zero_kernel, dim3(elementwise_grid(nk_el)), dim3(256), 0, stream, dk32, nk_el);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;

    const int64_t units = bh * m;
    if (units > 0 && n_q > 0 && n_k > 0) {
        const size_t sort_lds = ((size_t)(1 << tau) + kSortThreads) * 4;
        {
        KernelTimer timer("sort_kernel", stream);
        hipLaunchKernelGGL(sort_kernel, dim3((unsigned)(2 * units)), dim3(kSortThreads), sort_lds, stream, qcodes,
                           kcodes, units, n_q, n_k, tau, reinterpret_cast<int32_t *>(ws + L.qoff),
                           reinterpret_cast<int32_t *>(ws + L.koff), reinterpret_cast<uint16_t *>(ws + L.qperm),
                           reinterpret_cast<uint16_t *>(ws + L.kperm), reinterpret_cast<uint16_t *>(ws + L.qsorted),
                           reinterpret_cast<uint16_t *>(ws + L.ksorted));
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;

        PairArgs a;
        a.q = q; a.k = k; a.v = v; a.dy = dy;
        a.qoff = reinterpret_cast<const int32_t *>(ws + L.qoff);
        a.koff = reinterpret_cast<const int32_t *>(ws + L.koff);
        a.qperm = reinterpret_cast<const uint16_t *>(ws + L.qperm);
        a.kperm = reinterpret_cast<const uint16_t *>(ws + L.kperm);
        a.qsorted = reinterpret_cast<const uint16_t *>(ws + L.qsorted);
        a.ksorted = reinterpret_cast<const uint16_t *>(ws + L.ksorted);
        a.dq = dq32; a.dk = dk32;
        a.bh = bh; a.n_q = n_q; a.n_k = n_k; a.m = m; a.tau = tau;
        a.scale = (float)tau / (2.0f * (float)m);
        KernelTimer timer("pairs_kernel", stream);
        if (bf16)
            hipLaunchKernelGGL(pairs_kernel<true>, dim3((unsigned)units), dim3(kPairThreads), 0, stream, a);
        else
            hipLaunchKernelGGL(pairs_kernel<false>, dim3((unsigned)units), dim3(kPairThreads), 0, stream, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (bf16) {
        KernelTimer timer("to_bf16_kernel", stream);
        if (nq_el)
            hipLaunchKernelGGL(to_bf16_kernel, dim3(elementwise_grid(nq_el)), dim3(256), 0, stream, dq32,
                               static_cast<uint16_t *>(dq), nq_el);
        if (nk_el)
            hipLaunchKernelGGL(to_bf16_kernel, dim3(elementwise_grid(nk_el)), dim3(256), 0, stream, dk32,
                               static_cast<uint16_t *>(dk), nk_el);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace yoso
