// Backward dQ, dK of YOSO attention on MFMA (gfx950).
//
// Sec. 3.3, eq. (pseudo-gradient-q) evaluated on the sampled collisions:
//   dQ = tau/(2m) sum_h [(dY V^T) .* B_h] K,   dK = tau/(2m) sum_h [(dY V^T) .* B_h]^T Q.
// For one hash the nonzeros of B_h are blocks: query bucket c meets key bucket
// c.  Sorting the rows of Q and K by code turns B_h into a block-diagonal matrix
// in (sorted query, sorted key) coordinates.  This is the sum the paper writes as
// d runs of the table subroutine (eq. backward-d2), evaluated pair by pair: 3d
// multiply-adds per colliding pair instead of 2d^2 per row.
//
// The two outputs are the same computation with the roles swapped:
//   dQ_i = s sum_h sum_{j in bucket_h(i)} (dy_i . v_j) k_j
//   dK_j = s sum_h sum_{i in bucket_h(j)} (v_j . dy_i) q_i        (s = tau/(2m))
// so one "pass" routine serves both: rows x with row vectors a_x, partners y in
// the same bucket with vectors a'_y and b_y, out_x = s sum (a_x . a'_y) b_y.
//
// Kernels:
//   sort_kernel    one workgroup per (head, hash, side): histogram of the codes,
//                  exclusive scan -> bucket offsets, then row ids and codes in
//                  bucket order (a counting sort in LDS).
//   pass_kernel    one workgroup per (head, hash, side).  Each wave walks 16-row
//                  tiles of sorted rows; the partners that can collide with a tile
//                  form one contiguous range of sorted partners, visited 16 at a
//                  time:  S^T = A'_y A_x^T (16x16x32 MFMA), masked by code equality,
//                  out^T += B_y^T S^T (16x16x16 MFMA).  The finished tile is the
//                  hash's share of out for those rows; it is stored, not added,
//                  into a partial buffer [bh][n][m][64] (each row of each hash is
//                  written exactly once, so no atomics are needed).
//   reduce_kernel  out[b][x] = sum over the m hashes of the partial rows, in hash
//                  order (deterministic), written as fp32 or bf16.
// gfx950's global fp32 atomics sustain roughly 1.3 TB/s of payload, so a plain
// store of every partial plus one coalesced reduction beats accumulating with
// atomics.  Every fp32 product uses three fp16 MFMAs (hi*hi + hi*lo + lo*hi);
// the b vectors are scaled by 2^8 before splitting (undone on the way out).
#include "common.h"
#include "launch.h"
#include "timing.h"

namespace yoso {

namespace {

constexpr int kSortThreads = 256;
constexpr int kPassThreads = 256;
constexpr int kReduceThreads = 256;

// ---------------------------------------------------------------- counting sort
// codes are [bh][n][m]; unit = b*m + h reads column h with stride m.
__global__ __launch_bounds__(kSortThreads) void sort_kernel(const uint16_t *__restrict__ qcodes,
                                                            const uint16_t *__restrict__ kcodes, int m,
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
    const int64_t b = unit / m;
    const int h = static_cast<int>(unit - b * m);
    const int64_t n = kside ? n_k : n_q;
    const uint16_t *codes = (kside ? kcodes : qcodes) + b * n * m + h;
    int32_t *off = (kside ? koff : qoff) + unit * ((1 << tau) + 1);
    uint16_t *perm = (kside ? kperm : qperm) + unit * n;
    uint16_t *sorted = (kside ? ksorted : qsorted) + unit * n;
    const int B = 1 << tau;
    const int tid = threadIdx.x;

    for (int c = tid; c < B; c += kSortThreads) cnt[c] = 0;
    __syncthreads();
    for (int64_t i = tid; i < n; i += kSortThreads) atomicAdd(&cnt[codes[i * m] & (B - 1)], 1);
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
        const int c = codes[i * m] & (B - 1);
        const int32_t pos = atomicAdd(&cnt[c], 1);
        perm[pos] = static_cast<uint16_t>(i);
        sorted[pos] = static_cast<uint16_t>(c);
    }
}

// ---------------------------------------------------------------- pair passes
struct Side {
    const uint16_t *perm, *sorted;  // [units][n] rows in bucket order and their codes
    const int32_t *off;             // [units][2^tau + 1] bucket offsets
    int64_t n;
};

struct PassArgs {
    Side q, k;
    const void *qv, *kv, *vv, *dyv;  // Q, K, V, dY [bh][n][64]
    float *pq, *pk;                  // partials [bh][n][m][64]
    int64_t bh;
    int m, tau;
    float scale;                     // tau / (2m)
};

// out_x (for the 16 sorted rows of a tile) = scale * sum_{y in bucket(x)} (a_x . a'_y) b_y,
// stored at part[(row0 + x) * m + h][0:64].
template <bool BF16>
__device__ __forceinline__ void pass_run(const Side &rows, const Side &par, const void *a_row, const void *a_par,
                                         const void *b_par, float *part, int64_t unit, int64_t b, int h, int m,
                                         int tau, float scale) {
    const int nbk = (1 << tau) + 1;
    const uint16_t *rperm = rows.perm + unit * rows.n;
    const uint16_t *rsorted = rows.sorted + unit * rows.n;
    const int32_t *poff = par.off + unit * nbk;
    const uint16_t *pperm = par.perm + unit * par.n;
    const uint16_t *psorted = par.sorted + unit * par.n;
    const int64_t rrow0 = b * rows.n, prow0 = b * par.n;

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, c = lane & 15;
    const int64_t tiles = (rows.n + 15) >> 4;

    for (int64_t rt = wave; rt < tiles; rt += kPassThreads / 64) {
        const int64_t p0 = rt * 16;
        const int64_t plast = (p0 + 15 < rows.n) ? p0 + 15 : rows.n - 1;
        const int cfirst = rsorted[p0], clast = rsorted[plast];
        const int64_t pbeg = poff[cfirst], pend = poff[clast + 1];

        // row-side operand: a_x as the B operand of S^T (lane (g, c): row c, dims kb*32 + g*8 + [0,8))
        const bool rv_c = p0 + c < rows.n;
        const int64_t rrow_c = rv_c ? rrow0 + rperm[p0 + c] : 0;
        const int rcode_c = rv_c ? rsorted[p0 + c] : -2;
        floatx4 outT[4];
#pragma unroll
        for (int dt = 0; dt < 4; dt++) outT[dt] = floatx4{0.f, 0.f, 0.f, 0.f};

        if (pbeg < pend) {
            half8 ah[2], al[2];
#pragma unroll
            for (int kb = 0; kb < 2; kb++) {
                float t[8];
                if (rv_c) {
                    load8<BF16>(a_row, rrow_c * D + kb * 32 + g * 8, t);
                } else {
#pragma unroll
                    for (int i = 0; i < 8; i++) t[i] = 0.f;
                }
                split8(t, 1.0f, ah[kb], al[kb]);
            }
            for (int64_t y0 = pbeg; y0 < pend; y0 += 16) {
                // partner a'_y as the A operand of S^T (lane (g, c): partner c)
                const bool pv_c = y0 + c < pend;
                const int64_t prow_c = pv_c ? prow0 + pperm[y0 + c] : 0;
                half8 ph[2], pl[2];
#pragma unroll
                for (int kb = 0; kb < 2; kb++) {
                    float t[8];
                    if (pv_c) {
                        load8<BF16>(a_par, prow_c * D + kb * 32 + g * 8, t);
                    } else {
#pragma unroll
                        for (int i = 0; i < 8; i++) t[i] = 0.f;
                    }
                    split8(t, 1.0f, ph[kb], pl[kb]);
                }
                // partner b_y^T as A fragments of the output product:
                // lane (g, c) holds dims 16dt + c of partners y0 + 4g + [0,4)
                int pcode_r[4];
                int64_t prow_r[4];
                bool pv_r[4];
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const int64_t p = y0 + 4 * g + i;
                    pv_r[i] = p < pend;
                    prow_r[i] = pv_r[i] ? prow0 + pperm[p] : 0;
                    pcode_r[i] = pv_r[i] ? psorted[p] : -3;
                }
                half4 bh[4], bl[4];
#pragma unroll
                for (int dt = 0; dt < 4; dt++) {
                    float t[4];
#pragma unroll
                    for (int i = 0; i < 4; i++)
                        t[i] = pv_r[i] ? load1<BF16>(b_par, prow_r[i] * D + dt * 16 + c) : 0.f;
                    split4(t, 256.0f, bh[dt], bl[dt]);
                }
                // S^T[partner 4g+i][row c]
                floatx4 st = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kb = 0; kb < 2; kb++) st = mfma3_16x16x32(ph[kb], pl[kb], ah[kb], al[kb], st);
                float sv[4];
#pragma unroll
                for (int i = 0; i < 4; i++) sv[i] = (pcode_r[i] == rcode_c) ? st[i] * scale : 0.f;
                half4 sh, sl;
                split4(sv, 1.0f, sh, sl);
                // out^T[dim 16dt + 4g + i][row c] += sum_y b^T[dim][y] S^T[y][row]
#pragma unroll
                for (int dt = 0; dt < 4; dt++) outT[dt] = mfma3_16x16x16(bh[dt], bl[dt], sh, sl, outT[dt]);
            }
        }
        // lane (g, c) holds out[row c][dims 16dt + 4g + (0..3)]
        if (rv_c) {
            float *dst = part + ((rrow_c * m) + h) * D + 4 * g;
#pragma unroll
            for (int dt = 0; dt < 4; dt++) {
                const float4 o = make_float4(outT[dt][0] * (1.0f / 256.0f), outT[dt][1] * (1.0f / 256.0f),
                                             outT[dt][2] * (1.0f / 256.0f), outT[dt][3] * (1.0f / 256.0f));
                *reinterpret_cast<float4 *>(dst + dt * 16) = o;
            }
        }
    }
}

template <bool BF16>
__global__ __launch_bounds__(kPassThreads) void pass_kernel(PassArgs a) {
    const int64_t units = a.bh * a.m;
    const int64_t id = xcd_remap(blockIdx.x, 2 * units);
    const int64_t unit = id >> 1;
    const bool kside = id & 1;
    const int64_t b = unit / a.m;
    const int h = static_cast<int>(unit - b * a.m);
    if (!kside) {
        // dQ: rows = queries (a = dY), partners = keys (a' = V, b = K)
        pass_run<BF16>(a.q, a.k, a.dyv, a.vv, a.kv, a.pq, unit, b, h, a.m, a.tau, a.scale);
    } else {
        // dK: rows = keys (a = V), partners = queries (a' = dY, b = Q)
        pass_run<BF16>(a.k, a.q, a.vv, a.dyv, a.qv, a.pk, unit, b, h, a.m, a.tau, a.scale);
    }
}

// out[r][:] = sum_h part[r][h][:]; 16 lanes per row, 4 floats each.
template <bool BF16>
__global__ __launch_bounds__(kReduceThreads) void reduce_kernel(const float *__restrict__ part, void *__restrict__ out,
                                                                int64_t rows, int m) {
    const int64_t r = (static_cast<int64_t>(blockIdx.x) * kReduceThreads + threadIdx.x) >> 4;
    const int q = threadIdx.x & 15;
    if (r >= rows) return;
    const float4 *src = reinterpret_cast<const float4 *>(part + r * m * D) + q;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int h = 0; h < m; h++) {
        const float4 v = src[h * (D / 4)];
        s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
    }
    if constexpr (BF16) {
        uint2 o;
        o.x = static_cast<uint32_t>(f32_to_bf16(s.x)) | (static_cast<uint32_t>(f32_to_bf16(s.y)) << 16);
        o.y = static_cast<uint32_t>(f32_to_bf16(s.z)) | (static_cast<uint32_t>(f32_to_bf16(s.w)) << 16);
        reinterpret_cast<uint2 *>(static_cast<uint16_t *>(out) + r * D)[q] = o;
    } else {
        reinterpret_cast<float4 *>(static_cast<float *>(out) + r * D)[q] = s;
    }
}

__global__ void zero_kernel(float *__restrict__ p, int64_t count) {
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < count;
         e += static_cast<int64_t>(gridDim.x) * blockDim.x)
        p[e] = 0.f;
}

__global__ void zero_bf16_kernel(uint16_t *__restrict__ p, int64_t count) {
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < count;
         e += static_cast<int64_t>(gridDim.x) * blockDim.x)
        p[e] = 0;
}

unsigned elementwise_grid(int64_t count) {
    const int64_t blocks = (count + 255) / 256;
    return static_cast<unsigned>(blocks < 8192 ? (blocks > 0 ? blocks : 1) : 8192);
}

size_t align_up(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

template <bool BF16>
hipError_t launch_reduce(const float *part, void *out, int64_t rows, int m, hipStream_t stream) {
    if (rows == 0) return hipSuccess;
    const int64_t blocks = (rows * 16 + kReduceThreads - 1) / kReduceThreads;
    KernelTimer timer("reduce_kernel", stream);
    hipLaunchKernelGGL(reduce_kernel<BF16>, dim3(static_cast<unsigned>(blocks)), dim3(kReduceThreads), 0, stream,
                       part, out, rows, m);
    return hipGetLastError();
}

// Zero an output that no pair can reach (the other side is empty).
hipError_t zero_output(void *out, bool bf16, int64_t count, hipStream_t stream) {
    if (count == 0) return hipSuccess;
    KernelTimer timer("zero_kernel", stream);
    if (bf16)
        hipLaunchKernelGGL(zero_bf16_kernel, dim3(elementwise_grid(count)), dim3(256), 0, stream,
                           static_cast<uint16_t *>(out), count);
    else
        hipLaunchKernelGGL(zero_kernel, dim3(elementwise_grid(count)), dim3(256), 0, stream, static_cast<float *>(out),
                           count);
    return hipGetLastError();
}

}  // namespace

BackwardLayout backward_layout(bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m, int tau) {
    BackwardLayout L;
    const int64_t units = bh * m;
    const size_t nb = (static_cast<size_t>(1) << tau) + 1;
    size_t o = 0;
    L.qoff = o; o = align_up(o + units * nb * 4);
    L.koff = o; o = align_up(o + units * nb * 4);
    L.qperm = o; o = align_up(o + units * n_q * 2);
    L.kperm = o; o = align_up(o + units * n_k * 2);
    L.qsorted = o; o = align_up(o + units * n_q * 2);
    L.ksorted = o; o = align_up(o + units * n_k * 2);
    L.pq = o; o = align_up(o + static_cast<size_t>(bh) * n_q * m * D * 4);
    L.pk = o; o = align_up(o + static_cast<size_t>(bh) * n_k * m * D * 4);
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

    const int64_t units = bh * m;
    if (units == 0) return hipSuccess;
    if (n_q == 0 || n_k == 0) {
        // no pairs: dq and dk are zero
        if ((e = zero_output(dq, bf16, bh * n_q * D, stream)) != hipSuccess) return e;
        return zero_output(dk, bf16, bh * n_k * D, stream);
    }

    {
        const size_t sort_lds = (static_cast<size_t>(1 << tau) + kSortThreads) * 4;
        KernelTimer timer("sort_kernel", stream);
        hipLaunchKernelGGL(sort_kernel, dim3(static_cast<unsigned>(2 * units)), dim3(kSortThreads), sort_lds, stream,
                           qcodes, kcodes, m, n_q, n_k, tau, reinterpret_cast<int32_t *>(ws + L.qoff),
                           reinterpret_cast<int32_t *>(ws + L.koff), reinterpret_cast<uint16_t *>(ws + L.qperm),
                           reinterpret_cast<uint16_t *>(ws + L.kperm), reinterpret_cast<uint16_t *>(ws + L.qsorted),
                           reinterpret_cast<uint16_t *>(ws + L.ksorted));
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;

    PassArgs a;
    a.q = Side{reinterpret_cast<const uint16_t *>(ws + L.qperm), reinterpret_cast<const uint16_t *>(ws + L.qsorted),
               reinterpret_cast<const int32_t *>(ws + L.qoff), n_q};
    a.k = Side{reinterpret_cast<const uint16_t *>(ws + L.kperm), reinterpret_cast<const uint16_t *>(ws + L.ksorted),
               reinterpret_cast<const int32_t *>(ws + L.koff), n_k};
    a.qv = q; a.kv = k; a.vv = v; a.dyv = dy;
    a.pq = reinterpret_cast<float *>(ws + L.pq);
    a.pk = reinterpret_cast<float *>(ws + L.pk);
    a.bh = bh; a.m = m; a.tau = tau;
    a.scale = static_cast<float>(tau) / (2.0f * static_cast<float>(m));
    {
        KernelTimer timer("pass_kernel", stream);
        if (bf16)
            hipLaunchKernelGGL(pass_kernel<true>, dim3(static_cast<unsigned>(2 * units)), dim3(kPassThreads), 0,
                               stream, a);
        else
            hipLaunchKernelGGL(pass_kernel<false>, dim3(static_cast<unsigned>(2 * units)), dim3(kPassThreads), 0,
                               stream, a);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (bf16) {
        if ((e = launch_reduce<true>(a.pq, dq, bh * n_q, m, stream)) != hipSuccess) return e;
        return launch_reduce<true>(a.pk, dk, bh * n_k, m, stream);
    }
    if ((e = launch_reduce<false>(a.pq, dq, bh * n_q, m, stream)) != hipSuccess) return e;
    return launch_reduce<false>(a.pk, dk, bh * n_k, m, stream);
}

}  // namespace yoso
