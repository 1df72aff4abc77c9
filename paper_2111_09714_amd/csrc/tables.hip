// Bucket-table scatter/gather: the forward of YOSO attention and its dV.
//
// Sec. 3.2 overview: for one hash, a table H of 2^tau d-vectors receives
// H[f(k_j)] += v_j for every key, then query i reads H[f(q_i)].  Sec. 3.1:
// the output averages m hashes.  Remark 3: memory drops from O(m 2^tau d) to
// O(m 2^tau) by processing a few dimensions at a time -- which is exactly what
// makes the tables fit in LDS here.
//
//   forward:  src = key codes,   values = V,  dst = query codes -> Y
//   dV:       src = query codes, values = dY, dst = key codes   -> dV   (eq. gradient-v)
//
// Work split: one workgroup per (head, slice of DS feature dims).  It keeps the
// tables of G hashes for its DS dims in LDS, laid out [bucket][dim][hash] with
// the hash index fastest.  All m hashes fit at once for the shipped shapes
// (tau=8,m=32: DS=4; tau=8,m=16: DS=8; tau=9,m=32: DS=2; 128 KiB); otherwise
// hashes are processed in groups and the output is accumulated in fp32.
//
// Scatter: lane (h, key-slot) adds the DS values of one key into hash h's table
// with ds_add_f32.  Within a half-wave the 32 lanes hit 32 distinct banks
// (bank = (dim*G + h) mod 32; slots of different keys rotate their dims when
// G < 32).  Gather: lane (query, hash-lane) sums its share of hashes for the DS
// dims (hash and dim orders are rotated per query so the 32 lanes of a
// half-wave again hit distinct banks), then 8 lanes reduce with shuffles.
//
// Blocks of one head are placed on one XCD so that the DS-wide slices of the
// same value rows meet in one L2.
#include "common.h"
#include "launch.h"
#include "timing.h"

namespace yoso {

namespace {

constexpr int kTableThreads = 1024;

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
#pragma unroll
            for (int i = 0; i < DS; i++) v[i] = bf16_to_f32(p[i]);
        }
    } else {
        const float *p = static_cast<const float *>(base) + off;
        if constexpr (DS >= 4) {
#pragma unroll
            for (int c = 0; c < DS / 4; c++) {
                const float4 w = reinterpret_cast<const float4 *>(p)[c];
                v[4 * c] = w.x; v[4 * c + 1] = w.y; v[4 * c + 2] = w.z; v[4 * c + 3] = w.w;
            }
        } else if constexpr (DS == 2) {
            const float2 w = *reinterpret_cast<const float2 *>(p);
            v[0] = w.x; v[1] = w.y;
        } else {
            v[0] = p[0];
        }
    }
}

// out[s] = in[(s + rot) % DS]  (rot < DS), as a barrel of conditional moves.
template <int DS>
__device__ __forceinline__ void rotate(float v[DS], int rot) {
#pragma unroll
    for (int b = 1; b < DS; b <<= 1) {
        if (rot & b) {
            float t[DS];
#pragma unroll
            for (int s = 0; s < DS; s++) t[s] = v[(s + b) % DS];
#pragma unroll
            for (int s = 0; s < DS; s++) v[s] = t[s];
        }
    }
}

struct TableArgs {
    const uint16_t *src_codes;  // [bh][m][n_src]
    const void *values;         // [bh][n_src][64]
    const uint16_t *dst_codes;  // [bh][m][n_dst]
    void *out;                  // [bh][n_dst][64], dtype of values (final output)
    float *acc;                 // fp32 [bh][n_dst][64] running sum when several hash groups are needed
    int64_t bh, n_src, n_dst;
    int m, tau, G;              // G = hashes per LDS pass
    float scale;                // 1/m
};

template <bool BF16, int DS>
__global__ __launch_bounds__(kTableThreads) void table_kernel(TableArgs a) {
    extern __shared__ __align__(16) float tab[];  // [2^tau][DS][G]
    constexpr int S = D / DS;
    const int64_t blocks = a.bh * S;
    const int64_t logical = xcd_remap(blockIdx.x, blocks);
    const int64_t b = logical / S;
    const int slice = static_cast<int>(logical - b * S);
    const int G = a.G;
    const int buckets = 1 << a.tau;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    constexpr int nwaves = kTableThreads / 64;

    // scatter lane roles
    const int kpw = 64 / G;  // keys per wave step (G <= 64)
    const int sh = lane % G, skey = lane / G;
    const bool s_active = skey < kpw;
    const int srot = (G < 32) ? (skey % (32 / G)) % DS : 0;
    // gather lane roles
    const int gq = lane >> 3, ghs = lane & 7;
    const int U = (G + 7) >> 3;
    const int grot_l = (U < 4) ? ((gq / U) % DS) : 0;

    const int ngroups = (a.m + G - 1) / G;
    const int64_t vrow0 = b * a.n_src;
    const int64_t orow0 = b * a.n_dst;
    for (int grp = 0; grp < ngroups; grp++) {
        const int h0 = grp * G;
        const int gcount = min(G, a.m - h0);
        for (int e = tid; e < buckets * DS * G; e += kTableThreads) tab[e] = 0.f;
        __syncthreads();

        // ---- scatter: tab[c][l][h] += values[j][slice*DS + l]
        if (s_active && sh < gcount) {
            const uint16_t *codes = a.src_codes + (b * a.m + h0 + sh) * a.n_src;
            for (int64_t j = (int64_t)wave * kpw + skey; j < a.n_src; j += (int64_t)nwaves * kpw) {
                const int c = codes[j] & (buckets - 1);
                float v[DS];
                load_slice<BF16, DS>(a.values, (vrow0 + j) * D + slice * DS, v);
                rotate<DS>(v, srot);
                float *row = tab + (c * DS) * G + sh;
#pragma unroll
                for (int s = 0; s < DS; s++) {
                    const int l = (s + srot) % DS;
                    atomicAdd(row + l * G, v[s]);
                }
            }
        }
        __syncthreads();

        // ---- gather: out[i][slice*DS + l] (+)= scale * sum_h tab[code_h(i)][l][h]
        for (int64_t i0 = (int64_t)wave * 8; i0 < a.n_dst; i0 += (int64_t)nwaves * 8) {
            const int64_t i = i0 + gq;
            float acc[DS];
#pragma unroll
            for (int l = 0; l < DS; l++) acc[l] = 0.f;
            if (i < a.n_dst) {
                for (int u = 0; u < U; u++) {
                    const int h = ghs + 8 * ((u + gq) % U);
                    if (h < gcount) {
                        const int c = a.dst_codes[(b * a.m + h0 + h) * a.n_dst + i] & (buckets - 1);
                        const float *row = tab + (c * DS) * G + h;
#pragma unroll
                        for (int l = 0; l < DS; l++) acc[l] += row[((l + grot_l) % DS) * G];
                    }
                }
            }
            // reduce over the 8 hash lanes of this query
#pragma unroll
            for (int l = 0; l < DS; l++) {
                acc[l] += __shfl_xor(acc[l], 1);
                acc[l] += __shfl_xor(acc[l], 2);
                acc[l] += __shfl_xor(acc[l], 4);
            }
            // acc[l] holds dim (l + grot_l) % DS; lane ghs writes dims ghs, ghs+8, ...
            if (i < a.n_dst) {
#pragma unroll
                for (int d0 = 0; d0 < DS; d0 += 8) {
                    const int dim = d0 + ghs;
                    if (dim < DS) {
                        float val = 0.f;
#pragma unroll
                        for (int l = 0; l < DS; l++)
                            if ((l + grot_l) % DS == dim) val = acc[l];
                        val *= a.scale;
                        const int64_t off = (orow0 + i) * D + slice * DS + dim;
                        if (ngroups == 1) {
                            if constexpr (BF16)
                                static_cast<uint16_t *>(a.out)[off] = f32_to_bf16(val);
                            else
                                static_cast<float *>(a.out)[off] = val;
                        } else {
                            // the same lane owns this element in every group
                            a.acc[off] = (grp == 0) ? val : a.acc[off] + val;
                        }
                    }
                }
            }
        }
        __syncthreads();
    }
}

__global__ void f32_to_bf16_kernel(const float *__restrict__ in, uint16_t *__restrict__ out, int64_t count) {
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < count;
         e += (int64_t)gridDim.x * blockDim.x)
        out[e] = f32_to_bf16(in[e]);
}

template <bool BF16>
hipError_t launch_table_ds(int ds, const TableArgs &a, size_t lds, hipStream_t stream) {
    const int64_t blocks = a.bh * (D / ds);
    const dim3 grid((unsigned)blocks), block(kTableThreads);
    KernelTimer timer("table_kernel", stream);
    switch (ds) {
#define YOSO_CASE(X)                                                                      \
    case X:                                                                               \
        hipLaunchKernelGGL((table_kernel<BF16, X>), grid, block, lds, stream, a);         \
        break;
        YOSO_CASE(1) YOSO_CASE(2) YOSO_CASE(4) YOSO_CASE(8) YOSO_CASE(16)
#undef YOSO_CASE
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

TablePlan plan_table(int m, int tau) {
    TablePlan p;
    const size_t per_dim_hash = ((size_t)1 << tau) * 4;
    if (per_dim_hash * m <= kTableLdsBudget) {
        p.G = m;
        p.DS = 1;
        while (p.DS < kTableMaxDS && per_dim_hash * m * (p.DS * 2) <= kTableLdsBudget) p.DS *= 2;
    } else {
        p.DS = 1;
        p.G = (int)(kTableLdsBudget / per_dim_hash);
        if (p.G > m) p.G = m;
    }
    p.lds = per_dim_hash * p.G * p.DS;
    p.groups = (m + p.G - 1) / p.G;
    return p;
}

size_t table_workspace_bytes(bool bf16, int64_t bh, int64_t n_dst, int m, int tau) {
    const TablePlan p = plan_table(m, tau);
    if (p.groups > 1 && bf16) return (size_t)bh * n_dst * D * sizeof(float);
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
    a.scale = 1.0f / (float)m;
    hipError_t e = bf16 ? launch_table_ds<true>(p.DS, a, p.lds, stream) : launch_table_ds<false>(p.DS, a, p.lds, stream);
    if (e != hipSuccess) return e;
    if (p.groups > 1 && bf16) {
        const int64_t count = bh * n_dst * D;
        const int64_t blocks = (count + 255) / 256 < 4096 ? (count + 255) / 256 : 4096;
        KernelTimer timer("f32_to_bf16_kernel", stream);
        hipLaunchKernelGGL(f32_to_bf16_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a.acc,
                           static_cast<uint16_t *>(out), count);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace yoso
