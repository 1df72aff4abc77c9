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
// the same bucket with vectors a'_y and b_y, out_x = s sum_y (a_x . a'_y) b_y.
//
// Kernels:
//   sort_kernel    one workgroup per (head, hash, side): histogram of the codes,
//                  exclusive scan -> bucket offsets, then the rows in bucket order
//                  as packed entries (code << 16 | row) (a counting sort in LDS).
//   pass_kernel    one workgroup per (head, hash, side).  Each wave walks 16-row
//                  tiles of sorted rows; the partners that can collide with a tile
//                  form one contiguous range of sorted partners, visited 16 at a
//                  time:  S^T = A'_y A_x^T (16x16x32 MFMA), masked by code equality,
//                  out^T += B_y^T S^T (16x16x16 MFMA).  The partner rows of the next
//                  sub-tile are fetched while the current one computes; B_y is
//                  transposed through a per-wave LDS tile.  The finished tile is the
//                  hash's share of out for those rows; it is stored, not added, into a
//                  partial buffer [bh][n][m][64] (each row of each hash is written
//                  exactly once, so no atomics are needed).  Partials are fp32, or
//                  bf16 when the outputs are bf16.
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
constexpr int kPassWaves = kPassThreads / 64;
constexpr int kReduceThreads = 256;
constexpr int kTileStride = 2 * 64 + 8;  // halves per row of the per-wave transpose tile ([hi 64 | lo 64] + pad)
constexpr size_t kPassStageBudget = 24 * 1024;  // LDS bytes for staged partner entries + offsets

// ---------------------------------------------------------------- counting sort
// codes are [bh][n][m]; unit = b*m + h reads column h with stride m.
__global__ __launch_bounds__(kSortThreads) void sort_kernel(const uint16_t *__restrict__ qcodes,
                                                            const uint16_t *__restrict__ kcodes, int m,
                                                            int64_t n_q, int64_t n_k, int tau,
                                                            int32_t *__restrict__ qoff, int32_t *__restrict__ koff,
                                                            uint32_t *__restrict__ qent,
                                                            uint32_t *__restrict__ kent) {
    extern __shared__ int32_t cnt[];  // [buckets] counts, then cursors; + [kSortThreads] scan scratch
    int32_t *scan = cnt + (1 << tau);
    const int64_t unit = blockIdx.x >> 1;
    const bool kside = blockIdx.x & 1;
    const int64_t b = unit / m;
    const int h = static_cast<int>(unit - b * m);
    const int64_t n = kside ? n_k : n_q;
    const uint16_t *codes = (kside ? kcodes : qcodes) + b * n * m + h;
    int32_t *off = (kside ? koff : qoff) + unit * ((1 << tau) + 1);
    uint32_t *ent = (kside ? kent : qent) + unit * n;
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
        const uint32_t c = codes[i * m] & (B - 1);
        const int32_t pos = atomicAdd(&cnt[c], 1);
        ent[pos] = (c << 16) | static_cast<uint32_t>(i);
    }
}

// ---------------------------------------------------------------- pair passes
struct Side {
    const uint32_t *ent;  // [units][n] (code << 16 | row) in bucket order
    const int32_t *off;   // [units][2^tau + 1] bucket offsets
    int64_t n;
};

struct PassArgs {
    Side q, k;
    // Q, K, V, dY split into fp16 (hi, lo) pairs by split_kernel: row r holds 64 hi
    // halves then 64 lo halves; Q and K are scaled by 2^8 first
    const _Float16 *qs, *ks, *vs, *dys;
    void *pq, *pk;                   // partials [bh][n][m][64] (fp32, or bf16 for bf16 storage)
    int64_t bh;
    int m, tau;
    float scale;                     // tau / (2m)
};

// Operands of one 16-partner sub-tile (fp16 hi/lo halves).
struct PartnerRegs {
    half8 ah[2], al[2];  // a'_y of partner c: dims kb*32 + g*8 + [0,8), kb = 0, 1
    half8 bh[2], bl[2];  // b_y of partner c, same dims (transposed through LDS before use)
    int code_r[4];       // codes of partners 4g + i (negative past the range)
};

__device__ __forceinline__ half8 zero_if8(bool keep, half8 v) {
    return keep ? v : half8{0, 0, 0, 0, 0, 0, 0, 0};
}

// Loads are unconditional (a row of this head is always valid memory) and the
// values past the range are zeroed afterwards, so no branch sits between the
// issue of the loads and their use.
__device__ __forceinline__ void load_partners(PartnerRegs &r, const uint32_t *pent, int64_t y0, int64_t pend,
                                              int64_t prow0, const _Float16 *a_par, const _Float16 *b_par, int g,
                                              int c) {
    const bool ok = y0 + c < pend;
    const uint32_t e = pent[ok ? y0 + c : y0];
    const int64_t row = (prow0 + (e & 0xFFFFu)) * (2 * D);
#pragma unroll
    for (int kb = 0; kb < 2; kb++) {
        const int o = kb * 32 + g * 8;
        r.ah[kb] = zero_if8(ok, *reinterpret_cast<const half8 *>(a_par + row + o));
        r.al[kb] = zero_if8(ok, *reinterpret_cast<const half8 *>(a_par + row + D + o));
        r.bh[kb] = zero_if8(ok, *reinterpret_cast<const half8 *>(b_par + row + o));
        r.bl[kb] = zero_if8(ok, *reinterpret_cast<const half8 *>(b_par + row + D + o));
    }
#pragma unroll
    for (int i = 0; i < 4; i++) {
        const int64_t p = y0 + 4 * g + i;
        const bool in = p < pend;
        const uint32_t ei = pent[in ? p : y0];
        r.code_r[i] = in ? static_cast<int>(ei >> 16) : -3;
    }
}

// out^T += B_y^T S^T for one sub-tile held in r; ah/al are the row-side fragments.
__device__ __forceinline__ void compute_partners(const PartnerRegs &r, const half8 ah[2], const half8 al[2],
                                                 int rcode_c, float scale, _Float16 *tile, int g, int c,
                                                 floatx4 outT[4]) {
    // B_y through LDS: rows [partner][hi 64 | lo 64] halves; lane (g, c) then reads
    // partners 4g + i of dim 16dt + c
#pragma unroll
    for (int kb = 0; kb < 2; kb++) {
        *reinterpret_cast<half8 *>(tile + c * kTileStride + kb * 32 + g * 8) = r.bh[kb];
        *reinterpret_cast<half8 *>(tile + c * kTileStride + D + kb * 32 + g * 8) = r.bl[kb];
    }
    // the tile is private to this wave and LDS executes a wave's accesses in order:
    // only the compiler must keep the reads after the writes (and the next writes
    // after these reads)
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    half4 bh[4], bl[4];
#pragma unroll
    for (int dt = 0; dt < 4; dt++) {
#pragma unroll
        for (int i = 0; i < 4; i++) {
            bh[dt][i] = tile[(4 * g + i) * kTileStride + dt * 16 + c];
            bl[dt][i] = tile[(4 * g + i) * kTileStride + D + dt * 16 + c];
        }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    // S^T[partner 4g+i][row c]
    floatx4 st = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 2; kb++) st = mfma3_16x16x32(r.ah[kb], r.al[kb], ah[kb], al[kb], st);
    float sv[4];
#pragma unroll
    for (int i = 0; i < 4; i++) sv[i] = (r.code_r[i] == rcode_c) ? st[i] * scale : 0.f;
    half4 sh, sl;
    split4(sv, 1.0f, sh, sl);
#pragma unroll
    for (int dt = 0; dt < 4; dt++) outT[dt] = mfma3_16x16x16(bh[dt], bl[dt], sh, sl, outT[dt]);
}

template <bool BF16, bool STAGED>
__global__ __launch_bounds__(kPassThreads) void pass_kernel(PassArgs a) {
    extern __shared__ __align__(16) _Float16 smem[];
    _Float16 *tile = smem + (threadIdx.x >> 6) * (16 * kTileStride);  // per-wave transpose tile
    uint32_t *stage = reinterpret_cast<uint32_t *>(smem + kPassWaves * 16 * kTileStride);

    const int64_t units = a.bh * a.m;
    const int64_t id = xcd_remap(blockIdx.x, 2 * units);
    const int64_t unit = id >> 1;
    const bool kside = id & 1;
    const int64_t b = unit / a.m;
    const int h = static_cast<int>(unit - b * a.m);
    // dQ: rows = queries (a = dY), partners = keys (a' = V, b = K)
    // dK: rows = keys (a = V), partners = queries (a' = dY, b = Q)
    // (fields are selected by value: a runtime choice between references into the
    // kernel-argument struct would force a private copy of it)
    const int64_t n_r = kside ? a.k.n : a.q.n;
    const int64_t n_p = kside ? a.q.n : a.k.n;
    const uint32_t *r_ent = kside ? a.k.ent : a.q.ent;
    const uint32_t *p_ent = kside ? a.q.ent : a.k.ent;
    const int32_t *p_off = kside ? a.q.off : a.k.off;
    const _Float16 *a_row = kside ? a.vs : a.dys;
    const _Float16 *a_par = kside ? a.dys : a.vs;
    const _Float16 *b_par = kside ? a.qs : a.ks;
    void *part = kside ? a.pk : a.pq;

    const int nbk = (1 << a.tau) + 1;
    const uint32_t *rent = r_ent + unit * n_r;
    const uint32_t *pent = p_ent + unit * n_p;
    const int32_t *poff = p_off + unit * nbk;
    if constexpr (STAGED) {
        uint32_t *s_ent = stage;
        int32_t *s_off = reinterpret_cast<int32_t *>(stage + n_p);
        for (int64_t i = threadIdx.x; i < n_p; i += kPassThreads) s_ent[i] = pent[i];
        for (int i = threadIdx.x; i < nbk; i += kPassThreads) s_off[i] = poff[i];
        __syncthreads();
        pent = s_ent;
        poff = s_off;
    }
    const int64_t rrow0 = b * n_r, prow0 = b * n_p;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, c = lane & 15;
    const int64_t tiles = (n_r + 15) >> 4;

    uint32_t e_next = 0;
    if (wave < tiles && static_cast<int64_t>(wave) * 16 + c < n_r) e_next = rent[static_cast<int64_t>(wave) * 16 + c];
    for (int64_t t = wave; t < tiles; t += kPassWaves) {
        const uint32_t e = e_next;
        {
            const int64_t tn = t + kPassWaves;
            e_next = (tn < tiles && tn * 16 + c < n_r) ? rent[tn * 16 + c] : 0u;
        }
        const int64_t p0 = t * 16;
        const int nrow = static_cast<int>(n_r - p0 < 16 ? n_r - p0 : 16);
        const bool rv_c = c < nrow;
        const int rcode_c = rv_c ? static_cast<int>(e >> 16) : -2;
        const int64_t rrow_c = rrow0 + (e & 0xFFFFu);
        const int cfirst = static_cast<int>(__builtin_amdgcn_readlane(e, 0) >> 16);
        const int clast = static_cast<int>(__builtin_amdgcn_readlane(e, nrow - 1) >> 16);
        const int64_t pbeg = poff[cfirst], pend = poff[clast + 1];

        floatx4 outT[4];
#pragma unroll
        for (int dt = 0; dt < 4; dt++) outT[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
        if (pbeg < pend) {
            PartnerRegs A, B;
            load_partners(A, pent, pbeg, pend, prow0, a_par, b_par, g, c);
            half8 ah[2], al[2];
#pragma unroll
            for (int kb = 0; kb < 2; kb++) {
                const int o = kb * 32 + g * 8;
                ah[kb] = zero_if8(rv_c, *reinterpret_cast<const half8 *>(a_row + rrow_c * (2 * D) + o));
                al[kb] = zero_if8(rv_c, *reinterpret_cast<const half8 *>(a_row + rrow_c * (2 * D) + D + o));
            }
            for (int64_t y0 = pbeg;;) {
                if (y0 + 16 < pend) load_partners(B, pent, y0 + 16, pend, prow0, a_par, b_par, g, c);
                compute_partners(A, ah, al, rcode_c, a.scale, tile, g, c, outT);
                y0 += 16;
                if (y0 >= pend) break;
                if (y0 + 16 < pend) load_partners(A, pent, y0 + 16, pend, prow0, a_par, b_par, g, c);
                compute_partners(B, ah, al, rcode_c, a.scale, tile, g, c, outT);
                y0 += 16;
                if (y0 >= pend) break;
            }
        }
        // lane (g, c) holds out[row c][dims 16dt + 4g + (0..3)] * 256
        if (rv_c) {
            const int64_t base = ((rrow_c * a.m) + h) * D + 4 * g;
#pragma unroll
            for (int dt = 0; dt < 4; dt++) {
                const float4 o = make_float4(outT[dt][0] * (1.0f / 256.0f), outT[dt][1] * (1.0f / 256.0f),
                                             outT[dt][2] * (1.0f / 256.0f), outT[dt][3] * (1.0f / 256.0f));
                if constexpr (BF16) {
                    uint2 w;
                    w.x = static_cast<uint32_t>(f32_to_bf16(o.x)) | (static_cast<uint32_t>(f32_to_bf16(o.y)) << 16);
                    w.y = static_cast<uint32_t>(f32_to_bf16(o.z)) | (static_cast<uint32_t>(f32_to_bf16(o.w)) << 16);
                    *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(part) + base + dt * 16) = w;
                } else {
                    *reinterpret_cast<float4 *>(static_cast<float *>(part) + base + dt * 16) = o;
                }
            }
        }
    }
}

// Q, K, V, dY -> fp16 (hi, lo) rows [hi 64 | lo 64] for the pair passes; Q and K
// (the vectors that multiply S) are scaled by 2^8 so that their lo parts stay
// normal fp16 numbers.  One thread per 8 values.
template <bool BF16>
__global__ __launch_bounds__(256) void split_kernel(const void *__restrict__ q, const void *__restrict__ k,
                                                    const void *__restrict__ v, const void *__restrict__ dy,
                                                    _Float16 *__restrict__ qs, _Float16 *__restrict__ ks,
                                                    _Float16 *__restrict__ vs, _Float16 *__restrict__ dys,
                                                    int64_t rows_q, int64_t rows_k) {
    const int64_t per_q = rows_q * (D / 8), per_k = rows_k * (D / 8);
    const int64_t total = 2 * (per_q + per_k);
    for (int64_t tid = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; tid < total;
         tid += static_cast<int64_t>(gridDim.x) * 256) {
        // which: 0 = Q, 1 = dY (query side), 2 = K, 3 = V (key side)
        int which;
        int64_t t;
        if (tid < per_q) { which = 0; t = tid; }
        else if (tid < 2 * per_q) { which = 1; t = tid - per_q; }
        else if (tid < 2 * per_q + per_k) { which = 2; t = tid - 2 * per_q; }
        else { which = 3; t = tid - 2 * per_q - per_k; }
        const void *src = which == 0 ? q : which == 1 ? dy : which == 2 ? k : v;
        _Float16 *dst = which == 0 ? qs : which == 1 ? dys : which == 2 ? ks : vs;
        const float scale = (which == 0 || which == 2) ? 256.0f : 1.0f;
        const int64_t row = t / (D / 8);
        const int o = static_cast<int>(t - row * (D / 8)) * 8;
        float x[8];
        load8<BF16>(src, row * D + o, x);
        half8 hi, lo;
        split8(x, scale, hi, lo);
        *reinterpret_cast<half8 *>(dst + row * (2 * D) + o) = hi;
        *reinterpret_cast<half8 *>(dst + row * (2 * D) + D + o) = lo;
    }
}

// out[r][:] = sum_h part[r][h][:]; 16 lanes per row, 4 values each.
template <bool BF16>
__global__ __launch_bounds__(kReduceThreads) void reduce_kernel(const void *__restrict__ part, void *__restrict__ out,
                                                                int64_t rows, int m) {
    const int64_t r = (static_cast<int64_t>(blockIdx.x) * kReduceThreads + threadIdx.x) >> 4;
    const int q = threadIdx.x & 15;
    if (r >= rows) return;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if constexpr (BF16) {
        const uint2 *src = reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(part) + r * m * D) + q;
        for (int h = 0; h < m; h++) {
            const uint2 v = src[h * (D / 4)];
            s.x += __uint_as_float(v.x << 16);
            s.y += __uint_as_float(v.x & 0xFFFF0000u);
            s.z += __uint_as_float(v.y << 16);
            s.w += __uint_as_float(v.y & 0xFFFF0000u);
        }
        uint2 o;
        o.x = static_cast<uint32_t>(f32_to_bf16(s.x)) | (static_cast<uint32_t>(f32_to_bf16(s.y)) << 16);
        o.y = static_cast<uint32_t>(f32_to_bf16(s.z)) | (static_cast<uint32_t>(f32_to_bf16(s.w)) << 16);
        reinterpret_cast<uint2 *>(static_cast<uint16_t *>(out) + r * D)[q] = o;
    } else {
        const float4 *src = reinterpret_cast<const float4 *>(static_cast<const float *>(part) + r * m * D) + q;
        for (int h = 0; h < m; h++) {
            const float4 v = src[h * (D / 4)];
            s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
        }
        reinterpret_cast<float4 *>(static_cast<float *>(out) + r * D)[q] = s;
    }
}

__global__ void zero_kernel(uint32_t *__restrict__ p, int64_t count) {
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < count;
         e += static_cast<int64_t>(gridDim.x) * blockDim.x)
        p[e] = 0u;
}

unsigned elementwise_grid(int64_t count) {
    const int64_t blocks = (count + 255) / 256;
    return static_cast<unsigned>(blocks < 8192 ? (blocks > 0 ? blocks : 1) : 8192);
}

size_t align_up(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

template <bool BF16>
hipError_t launch_reduce(const void *part, void *out, int64_t rows, int m, hipStream_t stream) {
    if (rows == 0) return hipSuccess;
    const int64_t blocks = (rows * 16 + kReduceThreads - 1) / kReduceThreads;
    KernelTimer timer("reduce_kernel", stream);
    hipLaunchKernelGGL(reduce_kernel<BF16>, dim3(static_cast<unsigned>(blocks)), dim3(kReduceThreads), 0, stream,
                       part, out, rows, m);
    return hipGetLastError();
}

// Zero an output that no pair can reach (the other side is empty).  `bytes` is a
// multiple of 4 (rows of 64 fp32 or bf16 values).
hipError_t zero_output(void *out, int64_t bytes, hipStream_t stream) {
    const int64_t words = bytes / 4;
    if (words == 0) return hipSuccess;
    KernelTimer timer("zero_kernel", stream);
    hipLaunchKernelGGL(zero_kernel, dim3(elementwise_grid(words)), dim3(256), 0, stream, static_cast<uint32_t *>(out),
                       words);
    return hipGetLastError();
}

template <bool BF16>
hipError_t launch_pass(const PassArgs &a, int64_t units, hipStream_t stream) {
    const int64_t nmax = a.q.n > a.k.n ? a.q.n : a.k.n;
    const size_t stage = (static_cast<size_t>(nmax) + (static_cast<size_t>(1) << a.tau) + 1) * 4;
    const size_t tiles = static_cast<size_t>(kPassWaves) * 16 * kTileStride * 2;
    KernelTimer timer("pass_kernel", stream);
    if (stage <= kPassStageBudget)
        hipLaunchKernelGGL((pass_kernel<BF16, true>), dim3(static_cast<unsigned>(2 * units)), dim3(kPassThreads),
                           tiles + stage, stream, a);
    else
        hipLaunchKernelGGL((pass_kernel<BF16, false>), dim3(static_cast<unsigned>(2 * units)), dim3(kPassThreads),
                           tiles, stream, a);
    return hipGetLastError();
}

}  // namespace

BackwardLayout backward_layout(bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m, int tau) {
    BackwardLayout L;
    const int64_t units = bh * m;
    const size_t nb = (static_cast<size_t>(1) << tau) + 1;
    const size_t pbytes = bf16 ? 2 : 4;
    size_t o = 0;
    L.qoff = o; o = align_up(o + units * nb * 4);
    L.koff = o; o = align_up(o + units * nb * 4);
    L.qent = o; o = align_up(o + units * n_q * 4);
    L.kent = o; o = align_up(o + units * n_k * 4);
    L.qs = o; o = align_up(o + static_cast<size_t>(bh) * n_q * D * 4);
    L.dys = o; o = align_up(o + static_cast<size_t>(bh) * n_q * D * 4);
    L.ks = o; o = align_up(o + static_cast<size_t>(bh) * n_k * D * 4);
    L.vs = o; o = align_up(o + static_cast<size_t>(bh) * n_k * D * 4);
    L.pq = o; o = align_up(o + static_cast<size_t>(bh) * n_q * m * D * pbytes);
    L.pk = o; o = align_up(o + static_cast<size_t>(bh) * n_k * m * D * pbytes);
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
    const int64_t ebytes = bf16 ? 2 : 4;
    if (n_q == 0 || n_k == 0) {
        // no pairs: dq and dk are zero
        if ((e = zero_output(dq, bh * n_q * D * ebytes, stream)) != hipSuccess) return e;
        return zero_output(dk, bh * n_k * D * ebytes, stream);
    }

    {
        const size_t sort_lds = (static_cast<size_t>(1 << tau) + kSortThreads) * 4;
        KernelTimer timer("sort_kernel", stream);
        hipLaunchKernelGGL(sort_kernel, dim3(static_cast<unsigned>(2 * units)), dim3(kSortThreads), sort_lds, stream,
                           qcodes, kcodes, m, n_q, n_k, tau, reinterpret_cast<int32_t *>(ws + L.qoff),
                           reinterpret_cast<int32_t *>(ws + L.koff), reinterpret_cast<uint32_t *>(ws + L.qent),
                           reinterpret_cast<uint32_t *>(ws + L.kent));
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;

    _Float16 *qs = reinterpret_cast<_Float16 *>(ws + L.qs), *ks = reinterpret_cast<_Float16 *>(ws + L.ks);
    _Float16 *vs = reinterpret_cast<_Float16 *>(ws + L.vs), *dys = reinterpret_cast<_Float16 *>(ws + L.dys);
    {
        const int64_t threads = 2 * bh * (n_q + n_k) * (D / 8);
        const int64_t blocks = (threads + 255) / 256 < 65536 ? (threads + 255) / 256 : 65536;
        KernelTimer timer("split_kernel", stream);
        if (bf16)
            hipLaunchKernelGGL(split_kernel<true>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, q, k, v,
                               dy, qs, ks, vs, dys, bh * n_q, bh * n_k);
        else
            hipLaunchKernelGGL(split_kernel<false>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, q, k,
                               v, dy, qs, ks, vs, dys, bh * n_q, bh * n_k);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;

    PassArgs a;
    a.q = Side{reinterpret_cast<const uint32_t *>(ws + L.qent), reinterpret_cast<const int32_t *>(ws + L.qoff), n_q};
    a.k = Side{reinterpret_cast<const uint32_t *>(ws + L.kent), reinterpret_cast<const int32_t *>(ws + L.koff), n_k};
    a.qs = qs; a.ks = ks; a.vs = vs; a.dys = dys;
    a.pq = ws + L.pq;
    a.pk = ws + L.pk;
    a.bh = bh; a.m = m; a.tau = tau;
    a.scale = static_cast<float>(tau) / (2.0f * static_cast<float>(m));
    e = bf16 ? launch_pass<true>(a, units, stream) : launch_pass<false>(a, units, stream);
    if (e != hipSuccess) return e;
    if (bf16) {
        if ((e = launch_reduce<true>(a.pq, dq, bh * n_q, m, stream)) != hipSuccess) return e;
        return launch_reduce<true>(a.pk, dk, bh * n_k, m, stream);
    }
    if ((e = launch_reduce<false>(a.pq, dq, bh * n_q, m, stream)) != hipSuccess) return e;
    return launch_reduce<false>(a.pk, dk, bh * n_k, m, stream);
}

}  // namespace yoso
