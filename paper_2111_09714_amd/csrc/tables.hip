// Bucket-table scatter/gather: the forward of YOSO attention and its dV.
//
// Sec. 3.2 overview: for one hash, a table H of 2^tau d-vectors receives
// H[f(k_j)] += v_j for every key, then query i reads H[f(q_i)].  Sec. 3.1: the
// output averages the m hashes.  Remark 3: memory drops from O(m 2^tau d) to
// O(m 2^tau) by processing a few dimensions at a time, which is what lets the
// tables of every hash live in LDS at once here.
//
//   forward:  src = key codes,   values = V,  dst = query codes -> Y
//   dV:       src = query codes, values = dY, dst = key codes   -> dV   (eq. gradient-v)
//
// One workgroup per (head, slice of DS feature dims); it holds the tables of G
// hashes (all m for the shipped shapes) for its DS dims in LDS.
//
// Tables hold fixed-point integers, not floats: gfx950 executes LDS fp32
// atomic adds some 40x slower than integer ones, while a 64-bit integer add
// carries two values at once.  Each value v of the slice is quantised to
// q = rint(v 2^k) with one power-of-two scale per workgroup, chosen from the
// slice's largest |v| so that any bucket sum of up to n_src values stays below
// 2^30 in magnitude.  Two adjacent dims (q_lo, q_hi) are packed as the 64-bit
// integer q_hi 2^32 + q_lo; sums of packed words never corrupt each other's
// field because |sum q_lo| < 2^31.  Integer sums are exact and independent of
// the order of the atomics, so the tables (and the outputs) are deterministic.
// The only rounding is the quantisation, |error| <= 2^-k / 2 per value.
//
// LDS layout: word (c*G + h)*P + p holds dims (2p, 2p+1) of bucket c of hash
// h (P = DS/2 words per row).
//   scatter: one key per instruction; lane (h, p) adds its word of the key into
//            row (code_h, h).  The 32 lanes of a half-wave cover distinct
//            (h, p) in a row block whose stride is a multiple of the 64 LDS
//            banks, so they never conflict.
//   gather:  8 lanes per query, each reading the whole P-word rows of G/8
//            hashes in a rotated order (the 16 lanes of a 16-byte access pass
//            hit distinct bank groups), then a DPP butterfly sums the 8 lanes.
#include "common.h"
#include "launch.h"
#include "timing.h"

namespace yoso {

namespace {

constexpr int kTableThreads = 1024;
constexpr int kTableWaves = kTableThreads / 64;

template <bool BF16, int DS>
__device__ __forceinline__ void load_slice(const void *base, int64_t off, float v[DS]) {
    if constexpr (BF16) {
        const uint16_t *p = static_cast<const uint16_t *>(base) + off;
        if constexpr (DS >= 8) {
#pragma unroll
            for (int c = 0; c < DS / 8; c++) {
                const uint4 w = reinterpret_cast<const uint4 *>(p)[c];
                const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    v[c * 8 + 2 * i] = __uint_as_float(ws[i] << 16);
                    v[c * 8 + 2 * i + 1] = __uint_as_float(ws[i] & 0xFFFF0000u);
                }
            }
        } else if constexpr (DS == 4) {
            const uint2 w = *reinterpret_cast<const uint2 *>(p);
            v[0] = __uint_as_float(w.x << 16);
            v[1] = __uint_as_float(w.x & 0xFFFF0000u);
            v[2] = __uint_as_float(w.y << 16);
            v[3] = __uint_as_float(w.y & 0xFFFF0000u);
        } else {
            const uint32_t w = *reinterpret_cast<const uint32_t *>(p);
            v[0] = __uint_as_float(w << 16);
            v[1] = __uint_as_float(w & 0xFFFF0000u);
        }
    } else {
        const float *p = static_cast<const float *>(base) + off;
        if constexpr (DS >= 4) {
#pragma unroll
            for (int c = 0; c < DS / 4; c++) {
                const float4 w = reinterpret_cast<const float4 *>(p)[c];
                v[4 * c] = w.x; v[4 * c + 1] = w.y; v[4 * c + 2] = w.z; v[4 * c + 3] = w.w;
            }
        } else {
            const float2 w = *reinterpret_cast<const float2 *>(p);
            v[0] = w.x; v[1] = w.y;
        }
    }
}

struct TableArgs {
    const uint16_t *src_codes;  // [bh][n_src][m]
    const void *values;         // [bh][n_src][64]
    const uint16_t *dst_codes;  // [bh][n_dst][m]
    void *out;                  // [bh][n_dst][64], dtype of values
    float *acc;                 // fp32 running sums when the hashes take several LDS passes
    int64_t bh, n_src, n_dst;
    int m, tau, G;              // G = hashes per LDS pass
    int e_n;                    // ceil(log2(n_src)): bucket populations are < 2^e_n + 1
};

// (lo, hi) of a packed word whose fields are signed and |field sums| < 2^31.
__device__ __forceinline__ void unpack(unsigned long long w, int &lo, int &hi) {
    lo = static_cast<int>(static_cast<uint32_t>(w));
    hi = static_cast<int>(static_cast<long long>(w - static_cast<unsigned long long>(static_cast<long long>(lo))) >> 32);
}

template <bool BF16, int DS>
__global__ __launch_bounds__(kTableThreads) void table_kernel(TableArgs a) {
    constexpr int P = DS / 2;   // packed words per table row
    constexpr int S = D / DS;   // slices per head
    extern __shared__ __align__(16) unsigned long long tab[];  // [2^tau][G][P]
    __shared__ float wave_red[kTableWaves];
    __shared__ int scale_exp;

    const int64_t blocks = a.bh * S;
    const int64_t logical = xcd_remap(blockIdx.x, blocks);
    const int64_t b = logical / S;
    const int slice = static_cast<int>(logical - b * S);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int G = a.G;
    const int cmask = (1 << a.tau) - 1;
    const int64_t vbase = b * a.n_src * D + slice * DS;

    // ---- scale: largest |v| of this slice -> exponent k
    {
        float mx = 0.f;
        for (int64_t j = tid; j < a.n_src; j += kTableThreads) {
            float v[DS];
            load_slice<BF16, DS>(a.values, vbase + j * D, v);
#pragma unroll
            for (int d = 0; d < DS; d++) mx = fmaxf(mx, fabsf(v[d]));
        }
        mx = wave_max(mx);
        if (lane == 0) wave_red[wave] = mx;
        __syncthreads();
        if (tid == 0) {
            float t = 0.f;
            for (int w = 0; w < kTableWaves; w++) t = fmaxf(t, wave_red[w]);
            int k = 0;
            if (t > 0.f) {
                int ev;
                frexpf(t, &ev);  // t < 2^ev
                k = 30 - a.e_n - ev;
            }
            scale_exp = k;
        }
        __syncthreads();
    }
    const int k = scale_exp;

    // lane roles
    int GP = 1;
    while (GP < G) GP <<= 1;               // hashes rounded up to a power of two
    const int CPK = GP * P;                // (hash, word) combos per key
    const int KPI = CPK <= 64 ? 64 / CPK : 1;   // keys per instruction
    const int NI = CPK <= 64 ? 1 : CPK / 64;    // instructions per key (<= 2)
    const int slot = CPK <= 64 ? lane / CPK : 0;
    int sh[2], sp[2];
#pragma unroll
    for (int ii = 0; ii < 2; ii++) {
        const int combo = (CPK <= 64 ? lane % CPK : lane) + 64 * ii;
        sp[ii] = combo % P;
        sh[ii] = combo / P;
    }
    const int L = GP < 8 ? GP : 8;         // gather lanes per query
    const int HL = GP / L;                 // hashes per gather lane (<= 8)
    const int QPI = 64 / L;                // queries per gather instruction
    const int gq = lane / L, gr = lane % L;

    const int ngroups = (a.m + G - 1) / G;
    const int64_t src_row0 = b * a.n_src, dst_row0 = b * a.n_dst;
    const float inv_m = 1.0f / static_cast<float>(a.m);
    for (int grp = 0; grp < ngroups; grp++) {
        const int h0 = grp * G;
        const int gcount = min(G, a.m - h0);
        {
            const int words = (cmask + 1) * G * P;  // even
            ulonglong2 *t2 = reinterpret_cast<ulonglong2 *>(tab);
            for (int e = tid; e < words / 2; e += kTableThreads) t2[e] = make_ulonglong2(0ull, 0ull);
        }
        __syncthreads();

        // ---- scatter
        for (int64_t j0 = static_cast<int64_t>(wave) * 64; j0 < a.n_src; j0 += static_cast<int64_t>(kTableWaves) * 64) {
            // lane = key j0 + lane: quantised, packed words of its DS values
            uint32_t pw[2 * P];
            {
                const int64_t j = j0 + lane;
                float v[DS];
                if (j < a.n_src) {
                    load_slice<BF16, DS>(a.values, vbase + j * D, v);
                } else {
#pragma unroll
                    for (int d = 0; d < DS; d++) v[d] = 0.f;
                }
#pragma unroll
                for (int p = 0; p < P; p++) {
                    const int lo = __float2int_rn(ldexpf(v[2 * p], k));
                    const int hi = __float2int_rn(ldexpf(v[2 * p + 1], k));
                    const unsigned long long w = (static_cast<unsigned long long>(static_cast<uint32_t>(hi)) << 32) +
                                                 static_cast<unsigned long long>(static_cast<long long>(lo));
                    pw[2 * p] = static_cast<uint32_t>(w);
                    pw[2 * p + 1] = static_cast<uint32_t>(w >> 32);
                }
            }
            const int nk = static_cast<int>(a.n_src - j0 < 64 ? a.n_src - j0 : 64);
            const int nsteps = (nk + KPI - 1) / KPI;
            constexpr int B = 4;  // steps whose codes are fetched together
            for (int s0 = 0; s0 < nsteps; s0 += B) {
                int cc[B][2];
#pragma unroll
                for (int t = 0; t < B; t++) {
#pragma unroll
                    for (int ii = 0; ii < 2; ii++) {
                        const int key = (s0 + t) * KPI + slot;
                        const bool ok = ii < NI && s0 + t < nsteps && key < nk && sh[ii] < gcount;
                        cc[t][ii] = ok ? (a.src_codes[(src_row0 + j0 + key) * a.m + h0 + sh[ii]] & cmask) : -1;
                    }
                }
#pragma unroll
                for (int t = 0; t < B; t++) {
                    if (s0 + t >= nsteps) break;
                    const int kk = (s0 + t) * KPI;
                    uint32_t w[2 * P];
                    if (KPI == 1) {
#pragma unroll
                        for (int d = 0; d < 2 * P; d++) w[d] = __builtin_amdgcn_readlane(pw[d], kk);
                    } else if (KPI == 2) {
#pragma unroll
                        for (int d = 0; d < 2 * P; d++) {
                            const uint32_t w0 = __builtin_amdgcn_readlane(pw[d], kk);
                            const uint32_t w1 = __builtin_amdgcn_readlane(pw[d], kk + 1 < 64 ? kk + 1 : 63);
                            w[d] = slot ? w1 : w0;
                        }
                    } else {
#pragma unroll
                        for (int d = 0; d < 2 * P; d++) w[d] = __shfl(pw[d], (kk + slot) & 63);
                    }
#pragma unroll
                    for (int ii = 0; ii < 2; ii++) {
                        const int c = cc[t][ii];
                        if (c >= 0) {
                            uint32_t lo = w[0], hi = w[1];
#pragma unroll
                            for (int p = 1; p < P; p++) {
                                lo = sp[ii] == p ? w[2 * p] : lo;
                                hi = sp[ii] == p ? w[2 * p + 1] : hi;
                            }
                            const unsigned long long word = (static_cast<unsigned long long>(hi) << 32) | lo;
                            atomicAdd(&tab[(c * G + sh[ii]) * P + sp[ii]], word);
                        }
                    }
                }
            }
        }
        __syncthreads();

        // ---- gather: out[i][slice*DS + d] (+)= 2^-k / m * sum_h table[code_h(i)][h][d]
        for (int64_t i0 = static_cast<int64_t>(wave) * QPI; i0 < a.n_dst; i0 += static_cast<int64_t>(kTableWaves) * QPI) {
            const int64_t i = i0 + gq;
            const bool qok = i < a.n_dst;
            int cc[8], hh[8];
#pragma unroll
            for (int t = 0; t < 8; t++) {
                hh[t] = gr + L * ((t + gq) % (HL > 0 ? HL : 1));
                const bool ok = t < HL && qok && hh[t] < gcount;
                cc[t] = ok ? (a.dst_codes[(dst_row0 + i) * a.m + h0 + hh[t]] & cmask) : -1;
            }
            float acc[DS];
#pragma unroll
            for (int d = 0; d < DS; d++) acc[d] = 0.f;
#pragma unroll
            for (int t = 0; t < 8; t++) {
                if (cc[t] >= 0) {
                    const unsigned long long *row = tab + (cc[t] * G + hh[t]) * P;
                    unsigned long long wv[P];
                    if constexpr (P == 1) {
                        wv[0] = row[0];
                    } else {
#pragma unroll
                        for (int p = 0; p < P; p += 2) {
                            const ulonglong2 x = reinterpret_cast<const ulonglong2 *>(row)[p / 2];
                            wv[p] = x.x;
                            wv[p + 1] = x.y;
                        }
                    }
#pragma unroll
                    for (int p = 0; p < P; p++) {
                        int lo, hi;
                        unpack(wv[p], lo, hi);
                        acc[2 * p] += static_cast<float>(lo);
                        acc[2 * p + 1] += static_cast<float>(hi);
                    }
                }
            }
#pragma unroll
            for (int d = 0; d < DS; d++) acc[d] = group_sum(acc[d], L);
            if (qok) {
                const int64_t obase = (dst_row0 + i) * D + slice * DS;
#pragma unroll
                for (int d = 0; d < DS; d++) {
                    if (d % L != gr) continue;
                    const float v = ldexpf(acc[d], -k) * inv_m;
                    if (ngroups == 1) {
                        if constexpr (BF16)
                            static_cast<uint16_t *>(a.out)[obase + d] = f32_to_bf16(v);
                        else
                            static_cast<float *>(a.out)[obase + d] = v;
                    } else {
                        // the same lane owns this element in every group
                        const float prev = grp == 0 ? 0.f : a.acc[obase + d];
                        if (grp == ngroups - 1 && BF16)
                            static_cast<uint16_t *>(a.out)[obase + d] = f32_to_bf16(prev + v);
                        else
                            a.acc[obase + d] = prev + v;
                    }
                }
            }
        }
        __syncthreads();
    }
}

template <bool BF16>
hipError_t launch_table_ds(int ds, const TableArgs &a, size_t lds, hipStream_t stream) {
    const int64_t blocks = a.bh * (D / ds);
    const dim3 grid(static_cast<unsigned>(blocks)), block(kTableThreads);
    KernelTimer timer("table_kernel", stream);
    switch (ds) {
#define YOSO_CASE(X)                                                              \
    case X:                                                                       \
        hipLaunchKernelGGL((table_kernel<BF16, X>), grid, block, lds, stream, a); \
        break;
        YOSO_CASE(2) YOSO_CASE(4) YOSO_CASE(8) YOSO_CASE(16)
#undef YOSO_CASE
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

int ceil_log2(int64_t n) {
    int e = 0;
    while ((int64_t{1} << e) < n) e++;
    return e;
}

}  // namespace

TablePlan plan_table(int m, int tau) {
    TablePlan p;
    const size_t row_bytes_per_dim = (size_t{1} << tau) * 4;  // one int32 per bucket and dim
    if (row_bytes_per_dim * m * 2 <= kTableLdsBudget) {
        p.G = m;
        p.DS = 2;
        // widen the slice while the tables fit and a key still needs at most two instructions
        int gp = 1;
        while (gp < m) gp <<= 1;
        while (p.DS < kTableMaxDS && row_bytes_per_dim * m * (p.DS * 2) <= kTableLdsBudget && gp * p.DS <= 128)
            p.DS *= 2;
    } else {
        p.DS = 2;
        p.G = static_cast<int>(kTableLdsBudget / (row_bytes_per_dim * 2));
        if (p.G > m) p.G = m;
    }
    p.lds = row_bytes_per_dim * p.G * p.DS;
    p.groups = (m + p.G - 1) / p.G;
    return p;
}

size_t table_workspace_bytes(bool bf16, int64_t bh, int64_t n_dst, int m, int tau) {
    const TablePlan p = plan_table(m, tau);
    if (p.groups > 1 && bf16) return static_cast<size_t>(bh) * n_dst * D * sizeof(float);
    return 0;
}

hipError_t launch_table(const uint16_t *src_codes, const void *values, const uint16_t *dst_codes, void *out,
                        bool bf16, int64_t bh, int64_t n_src, int64_t n_dst, int m, int tau, void *workspace,
                        hipStream_t stream) {
    if (bh == 0 || n_dst == 0) return hipSuccess;
    const TablePlan p = plan_table(m, tau);
    TableArgs a;
    a.src_codes = src_codes;
    a.values = values;
    a.dst_codes = dst_codes;
    a.out = out;
    a.acc = (p.groups > 1) ? (bf16 ? static_cast<float *>(workspace) : static_cast<float *>(out)) : nullptr;
    a.bh = bh;
    a.n_src = n_src;
    a.n_dst = n_dst;
    a.m = m;
    a.tau = tau;
    a.G = p.G;
    a.e_n = ceil_log2(n_src);
    return bf16 ? launch_table_ds<true>(p.DS, a, p.lds, stream) : launch_table_ds<false>(p.DS, a, p.lds, stream);
}

}  // namespace yoso
