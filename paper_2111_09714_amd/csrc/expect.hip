// YOSO-E: the exact expectation of YOSO over the hash functions (gfx950).
//
// Sec. 4 (YOSO-E: "the expected attention weights are directly computed using
// collision probability", the limit of infinitely many hashes) with the collision
// probability of eq. yoso-expectation / the Fig. 2 caption:
//   P_ij = (1 - arccos(cos(q_i, k_j)) / pi)^tau
//   Y  = P V                                   (the limit of the sampled forward)
//   dV = P^T dY                                (eq. gradient-v in expectation)
//   dQ = (tau/2) [(dY V^T) .* P] K             (eq. pseudo-gradient-q in expectation)
//   dK = (tau/2) [(dY V^T) .* P]^T Q           (its symmetric form)
// These are the expectations of the sampled forward and of the sampled surrogate
// backward, so YOSO-E is what YOSO tends to as m grows.
//
// Flash-style dense tiles on MFMA.  A workgroup (4 waves x 16 rows) keeps 64
// "fixed" rows R in registers and streams the other side C through LDS in tiles
// of 64 rows.  Per 16 x 16 block: S^T = x_C x_R^T (cosines, 16x16x32 f16 MFMA with
// fp16 (hi, lo) operands, three products), an elementwise arccos-power, and
// out_R^T += Y_C^T W for one or two weightings W (16x16x16 MFMA, three products).
// Three instantiations:
//   forward : R = queries, C = keys;    W1 = P                -> Y  (Y_C = V)
//   bwd_kv  : R = keys,    C = queries; W1 = P                -> dV (Y_C = dY)
//                                       W2 = (tau/2) G .* P   -> dK (Y_C = Q),
//             G = V_R dY_C^T
//   bwd_q   : R = queries, C = keys;    W2 = (tau/2) G .* P   -> dQ (Y_C = K),
//             G = dY_R V_C^T
// Scaling for the fp16 pairs, so that hi and lo stay normal fp16 numbers whatever
// the data's magnitude (all scales powers of two, divided out in fp32):
//   cosine rows: normalised, times 2^8;
//   fixed G rows (V in bwd_kv, dY in bwd_q): each row by 2^(13 - e), max|row| < 2^e;
//   streamed data rows (G rows, summed rows): each 64-row tile by 2^(13 - e), e from
//   the tile's largest |value|; the accumulators are rescaled (exactly, by a power
//   of two) whenever a tile's scale differs from the previous one;
//   weights: P by 2^15 and (tau/2) G P by 2^-k_tau, both then below 2^15.
#include "common.h"
#include "launch.h"
#include "timing.h"

namespace yoso {

namespace {

constexpr int kExpThreads = 256;
constexpr int kExpRows = 64;   // fixed rows per workgroup (16 per wave)
constexpr int kExpTile = 64;   // streamed rows per LDS tile
constexpr float kUnitScale = 256.0f;  // cosine rows: unit length times 2^8
constexpr float kPScale = 32768.0f;   // P weights: P 2^15 <= 2^15

enum : int { kExpFwd = 0, kExpBwdKV = 1, kExpBwdQ = 2 };

struct ExpArgs {
    const void *xr, *ar;            // fixed side: rows whose cosines are taken; rows of G (bwd)
    const void *xc, *bc, *yc;       // streamed side: cosine rows; G rows (bwd); rows that are summed
    void *out1, *out2;              // P-weighted sum (fwd, bwd_kv); G-weighted sum (bwd)
    int64_t bh;
    int n_r, n_c, tau;
};

// 16-byte chunk `chunk` (0..15) of row `row` in a tile of 256-byte rows, XOR-swizzled
// so that 16 rows read at one chunk, and 4 rows read at 2 chunks (the transpose
// reads), fall on distinct banks.
__device__ __forceinline__ uint32_t xswz(int row, int chunk) {
    const int f = ((2 * row + ((row >> 2) & 1)) & 15) ^ ((row >> 3) & 1);
    return static_cast<uint32_t>(row * 256 + ((chunk ^ f) << 4));
}

__device__ __forceinline__ half4 xtr_load(const unsigned char *p) {
    typedef short short4v __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) short4v lds_short4;
    return __builtin_bit_cast(half4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4 *)(p)));
}

// collision probability of two rows with cosine c: (1 - arccos(c)/pi)^tau
__device__ __forceinline__ float collision_p(float c, int tau) {
    c = fminf(fmaxf(c, -1.0f), 1.0f);
    const float base = 1.0f - acosf(c) * 0.31830988618379067f;
    float r = 1.0f, b = base;
    for (int e = tau; e; e >>= 1) {  // tau is uniform
        if (e & 1) r *= b;
        b *= b;
    }
    return r;
}

template <bool BF16, int MODE>
__global__ __launch_bounds__(kExpThreads, 2) void expect_kernel(ExpArgs a) {
    constexpr bool kP = MODE != kExpBwdQ;  // a P-weighted output
    constexpr bool kG = MODE != kExpFwd;   // a G-weighted output
    // streamed tile: cosine rows (unit, scaled 2^8), G rows / bwd_kv's summed rows
    // (scaled 2^4), summed rows (scaled 2^4); [row][hi 64 | lo 64] halves, swizzled
    __shared__ __align__(16) unsigned char xc_lds[kExpTile * 256];
    __shared__ __align__(16) unsigned char bc_lds[kG ? kExpTile * 256 : 16];
    __shared__ __align__(16) unsigned char yc_lds[kExpTile * 256];
    __shared__ float tmax[8];  // the waves' largest |value| of the staged G rows and summed rows

    const int64_t tiles_r = (a.n_r + kExpRows - 1) / kExpRows;
    const int64_t blk = xcd_remap(blockIdx.x, a.bh * tiles_r);
    const int64_t b = blk / tiles_r;
    const int r0 = static_cast<int>(blk - b * tiles_r) * kExpRows;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c = lane & 15;

    // ---- fixed rows in MFMA operand layout: lane (g, c) holds row c of the wave's
    // 16, dims kb*32 + 8g + [0, 8)
    const int rrow = r0 + wave * 16 + c;
    const int rcl = min(rrow, a.n_r - 1);  // rows past the end read the last row, never stored
    half8 xrh[2], xrl[2], arh[2], arl[2];
    int ea = 0;  // the lane's G row is scaled by 2^(13 - ea)
    {
        float x[2][8];
        const int64_t off = (b * a.n_r + rcl) * D;
        load8<BF16>(a.xr, off + 8 * g, x[0]);
        load8<BF16>(a.xr, off + 32 + 8 * g, x[1]);
        float ss = 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; kb++)
#pragma unroll
            for (int i = 0; i < 8; i++) ss += x[kb][i] * x[kb][i];
        // the row's other three quarters sit in lanes c + 16, c + 32, c + 48
        ss += __shfl_xor(ss, 16);
        ss += __shfl_xor(ss, 32);
        const float inv = ss > 0.f ? kUnitScale / sqrtf(ss) : 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; kb++) split8(x[kb], inv, xrh[kb], xrl[kb]);
        if constexpr (kG) {
            float y[2][8];
            load8<BF16>(a.ar, off + 8 * g, y[0]);
            load8<BF16>(a.ar, off + 32 + 8 * g, y[1]);
            float mx = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; kb++)
#pragma unroll
                for (int i = 0; i < 8; i++) mx = fmaxf(mx, fabsf(y[kb][i]));
            mx = fmaxf(mx, __shfl_xor(mx, 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            ea = pow2_above(mx);
#pragma unroll
            for (int kb = 0; kb < 2; kb++) split8(y[kb], ldexpf(1.0f, 13 - ea), arh[kb], arl[kb]);
        }
    }

    floatx4 out1[4], out2[4];
#pragma unroll
    for (int dt = 0; dt < 4; dt++) out1[dt] = out2[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
    const floatx4 z4 = {0.f, 0.f, 0.f, 0.f};
    const float half_tau = 0.5f * static_cast<float>(a.tau);
    const int pr = 4 * g + (c >> 2), a4 = c & 3;

    // tile loading: lane l of wave w stages streamed row 16w + (l & 15), dims
    // 16 (l >> 4) + [0, 16): the 16 lanes of a quarter-wave write 16 rows at one
    // chunk, which the swizzle puts on distinct banks (with 4 rows x 4 chunks per
    // quarter-wave, rows 0-3 would land on one set of 4 chunks)
    const int lrow = 16 * wave + (lane & 15), lq = lane >> 4;
    // this lane's 16 values of streamed row c0 + lrow (0 past the end) and their max |.|
    auto load_row = [&](const void *src, int c0, float x[16]) {
        const int row = c0 + lrow;
        const int64_t off = (b * a.n_c + min(row, a.n_c - 1)) * D + 16 * lq;
        load8<BF16>(src, off, x);
        load8<BF16>(src, off + 8, x + 8);
        const bool ok = row < a.n_c;
        float mx = 0.f;
#pragma unroll
        for (int i = 0; i < 16; i++) {
            x[i] = ok ? x[i] : 0.f;
            mx = fmaxf(mx, fabsf(x[i]));
        }
        return mx;
    };
    auto put_row = [&](unsigned char *dst, const float x[16], float scale) {
        half8 h[2], l[2];
        split8(x, scale, h[0], l[0]);
        split8(x + 8, scale, h[1], l[1]);
#pragma unroll
        for (int u = 0; u < 2; u++) {
            *reinterpret_cast<half8 *>(dst + xswz(lrow, 2 * lq + u)) = h[u];
            *reinterpret_cast<half8 *>(dst + xswz(lrow, 8 + 2 * lq + u)) = l[u];
        }
    };
    // cosine rows, normalised (the row's four threads are lanes l, l^16, l^32, l^48)
    auto stage_unit = [&](unsigned char *dst, const void *src, int c0) {
        float x[16];
        load_row(src, c0, x);
        float ss = 0.f;
#pragma unroll
        for (int i = 0; i < 16; i++) ss += x[i] * x[i];
        ss += __shfl_xor(ss, 16);
        ss += __shfl_xor(ss, 32);
        put_row(dst, x, ss > 0.f ? kUnitScale / sqrtf(ss) : 0.f);
    };
    // A-operand rows of sub-block cb (lane (g, c): row 16cb + c, dims kb*32 + 8g + [0, 8))
    auto read_rows = [&](const unsigned char *t, int cb, half8 h[2], half8 l[2]) {
#pragma unroll
        for (int kb = 0; kb < 2; kb++) {
            h[kb] = *reinterpret_cast<const half8 *>(t + xswz(16 * cb + c, kb * 4 + g));
            l[kb] = *reinterpret_cast<const half8 *>(t + xswz(16 * cb + c, 8 + kb * 4 + g));
        }
    };
    // transposed rows of sub-block cb as a 16x16x16 A operand (lane (g, c): dim
    // 16dt + c, rows 16cb + 4g .. +3)
    auto read_rows_t = [&](const unsigned char *t, int cb, half4 h[4], half4 l[4]) {
#pragma unroll
        for (int dt = 0; dt < 4; dt++) {
            h[dt] = xtr_load(t + xswz(16 * cb + pr, 2 * dt + (a4 >> 1)) + 8 * (a4 & 1));
            l[dt] = xtr_load(t + xswz(16 * cb + pr, 8 + 2 * dt + (a4 >> 1)) + 8 * (a4 & 1));
        }
    };
    auto sdot = [&](const half8 ah[2], const half8 al[2], const half8 bh[2], const half8 bl[2]) {
        floatx4 s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[0], bh[0], z4, 0, 0, 0);
        floatx4 s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[1], bh[1], z4, 0, 0, 0);
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[0], bl[0], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[1], bl[1], s1, 0, 0, 0);
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[0], bh[0], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[1], bh[1], s1, 0, 0, 0);
        return s0 + s1;
    };
    auto accum = [&](floatx4 out[4], const half4 yh[4], const half4 yl[4], const float w[4]) {
        half4 wh, wl;
        split4(w, 1.0f, wh, wl);
#pragma unroll
        for (int dt = 0; dt < 4; dt++) out[dt] = __builtin_amdgcn_mfma_f32_16x16x16f16(yh[dt], wh, out[dt], 0, 0, 0);
#pragma unroll
        for (int dt = 0; dt < 4; dt++) out[dt] = __builtin_amdgcn_mfma_f32_16x16x16f16(yh[dt], wl, out[dt], 0, 0, 0);
#pragma unroll
        for (int dt = 0; dt < 4; dt++) out[dt] = __builtin_amdgcn_mfma_f32_16x16x16f16(yl[dt], wh, out[dt], 0, 0, 0);
    };

    // tile exponents of the streamed data rows (G rows bc, summed rows yc) of the
    // tile whose products the accumulators hold
    int eb = 0, ey = 0;
    // (tau/2) G P is scaled by 2^-ktau: |G| < 2^32 after the row and tile scalings
    // (both sides' norms below 2^16), so the weight stays below 2^15
    int ktau = 0;
    while ((1 << ktau) < a.tau) ktau++;  // 2^ktau >= tau, i.e. 2^(ktau-1) >= tau/2
    const float wg = half_tau * ldexpf(1.0f, -(17 + ktau - 1));
    for (int c0 = 0; c0 < a.n_c; c0 += kExpTile) {
        __syncthreads();  // the previous tile has been read, and its maxima
        stage_unit(xc_lds, a.xc, c0);
        float xb[16], xy[16];
        float mb = 0.f;
        if constexpr (kG) mb = load_row(a.bc, c0, xb);
        float my = load_row(a.yc, c0, xy);
        mb = wave_max(mb);
        my = wave_max(my);
        if (lane == 0) {
            tmax[wave] = mb;
            tmax[4 + wave] = my;
        }
        __syncthreads();
        const int eb_new = pow2_above(fmaxf(fmaxf(tmax[0], tmax[1]), fmaxf(tmax[2], tmax[3])));
        const int ey_new = pow2_above(fmaxf(fmaxf(tmax[4], tmax[5]), fmaxf(tmax[6], tmax[7])));
        if constexpr (kG) put_row(bc_lds, xb, ldexpf(1.0f, 13 - eb_new));
        put_row(yc_lds, xy, ldexpf(1.0f, 13 - ey_new));
        // bring the sums so far to this tile's scales (exact power-of-two factors)
        if (c0 > 0) {
            const int e1o = MODE == kExpFwd ? ey : eb, e1n = MODE == kExpFwd ? ey_new : eb_new;
            const float f1 = ldexpf(1.0f, e1o - e1n), f2 = ldexpf(1.0f, eb + ey - eb_new - ey_new);
#pragma unroll
            for (int dt = 0; dt < 4; dt++) {
                if constexpr (kP) out1[dt] *= f1;
                if constexpr (kG) out2[dt] *= f2;
            }
        }
        eb = eb_new;
        ey = ey_new;
        __syncthreads();
#pragma unroll 1
        for (int cb = 0; cb < kExpTile / 16; cb++) {
            if (c0 + 16 * cb >= a.n_c) break;
            half8 xch[2], xcl[2];
            read_rows(xc_lds, cb, xch, xcl);
            // S^T block: lane (g, c) = cos(C row 16cb + 4g + i, R row c), scaled 2^16
            const floatx4 st = sdot(xch, xcl, xrh, xrl);
            float p[4];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const bool ok = c0 + 16 * cb + 4 * g + i < a.n_c;
                p[i] = ok ? collision_p(st[i] * (1.0f / (kUnitScale * kUnitScale)), a.tau) : 0.f;
            }
            if constexpr (kP) {
                // P 2^15 against the P-summed rows (V forward, dY in bwd_kv)
                float w[4];
#pragma unroll
                for (int i = 0; i < 4; i++) w[i] = p[i] * kPScale;
                half4 yh[4], yl[4];
                read_rows_t(MODE == kExpFwd ? yc_lds : bc_lds, cb, yh, yl);
                accum(out1, yh, yl, w);
            }
            if constexpr (kG) {
                half8 bh[2], bl[2];
                read_rows(bc_lds, cb, bh, bl);
                // G^T block: lane (g, c) = (b_C row 16cb + 4g + i) . (a_R row c), scaled
                // 2^(13 - eb) 2^(13 - ea)
                const floatx4 gt = sdot(bh, bl, arh, arl);
                float w[4];
#pragma unroll
                for (int i = 0; i < 4; i++) w[i] = gt[i] * p[i] * wg;
                half4 yh[4], yl[4];
                read_rows_t(yc_lds, cb, yh, yl);
                accum(out2, yh, yl, w);
            }
        }
    }

    // ---- the fixed rows' outputs: lane (g, c) holds out[R row c][16dt + 4g + i]
    if (rrow < a.n_r) {
        auto put = [&](void *dst, const floatx4 o[4], float sc) {
#pragma unroll
            for (int dt = 0; dt < 4; dt++) {
                const int64_t off = (b * a.n_r + rrow) * D + 16 * dt + 4 * g;
                if constexpr (BF16) {
                    uint2 w;
                    w.x = static_cast<uint32_t>(f32_to_bf16(o[dt][0] * sc)) |
                          (static_cast<uint32_t>(f32_to_bf16(o[dt][1] * sc)) << 16);
                    w.y = static_cast<uint32_t>(f32_to_bf16(o[dt][2] * sc)) |
                          (static_cast<uint32_t>(f32_to_bf16(o[dt][3] * sc)) << 16);
                    *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(dst) + off) = w;
                } else {
                    *reinterpret_cast<float4 *>(static_cast<float *>(dst) + off) =
                        make_float4(o[dt][0] * sc, o[dt][1] * sc, o[dt][2] * sc, o[dt][3] * sc);
                }
            }
        };
        // out1 = P 2^15 x (summed rows 2^(13 - e1)); out2 = (tau/2) G P 2^-ktau' x
        // (G rows 2^(13 - eb)) (fixed G row 2^(13 - ea)) x (summed rows 2^(13 - ey))
        const int e1 = MODE == kExpFwd ? ey : eb;
        if constexpr (kP) put(a.out1, out1, ldexpf(1.0f / kPScale, e1 - 13));
        if constexpr (kG) put(a.out2, out2, ldexpf(1.0f, (17 + ktau - 1) + eb - 13 + ea - 13 + ey - 13));
    }
}

__global__ void expect_zero_kernel(uint32_t *__restrict__ p, int64_t words) {
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < words;
         e += static_cast<int64_t>(gridDim.x) * blockDim.x)
        p[e] = 0u;
}

// zero `bytes` (a multiple of 4) of an output that no pair reaches
hipError_t zero_rows_async(void *p, int64_t bytes, hipStream_t stream) {
    const int64_t words = bytes / 4;
    if (words == 0) return hipSuccess;
    const int64_t blocks = (words + 255) / 256;
    hipLaunchKernelGGL(expect_zero_kernel, dim3(static_cast<unsigned>(blocks < 4096 ? blocks : 4096)), dim3(256), 0,
                       stream, static_cast<uint32_t *>(p), words);
    return hipGetLastError();
}

template <bool BF16, int MODE>
hipError_t launch_mode(const ExpArgs &a, hipStream_t stream, const char *name) {
    const int64_t blocks = a.bh * ((a.n_r + kExpRows - 1) / kExpRows);
    if (blocks == 0) return hipSuccess;
    KernelTimer timer(name, stream);
    hipLaunchKernelGGL((expect_kernel<BF16, MODE>), dim3(static_cast<unsigned>(blocks)), dim3(kExpThreads), 0, stream,
                       a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_expect_forward(const void *q, const void *k, const void *v, void *y, bool bf16, int64_t bh,
                                 int64_t n_q, int64_t n_k, int tau, hipStream_t stream) {
    if (bh == 0 || n_q == 0) return hipSuccess;
    if (n_k == 0) return zero_rows_async(y, bh * n_q * D * (bf16 ? 2 : 4), stream);
    ExpArgs a{};
    a.xr = q; a.xc = k; a.yc = v; a.out1 = y;
    a.bh = bh; a.n_r = static_cast<int>(n_q); a.n_c = static_cast<int>(n_k); a.tau = tau;
    return bf16 ? launch_mode<true, kExpFwd>(a, stream, "expect_fwd_kernel")
                : launch_mode<false, kExpFwd>(a, stream, "expect_fwd_kernel");
}

hipError_t launch_expect_backward(const void *q, const void *k, const void *v, const void *dy, void *dq, void *dk,
                                  void *dv, bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int tau,
                                  hipStream_t stream) {
    if (bh == 0) return hipSuccess;
    const int64_t e = bf16 ? 2 : 4;
    hipError_t err;
    if (n_q == 0 || n_k == 0) {
        if ((err = zero_rows_async(dq, bh * n_q * D * e, stream)) != hipSuccess) return err;
        if ((err = zero_rows_async(dk, bh * n_k * D * e, stream)) != hipSuccess) return err;
        return zero_rows_async(dv, bh * n_k * D * e, stream);
    }
    // keys fixed, queries streamed: dV and dK
    ExpArgs a{};
    a.xr = k; a.ar = v; a.xc = q; a.bc = dy; a.yc = q; a.out1 = dv; a.out2 = dk;
    a.bh = bh; a.n_r = static_cast<int>(n_k); a.n_c = static_cast<int>(n_q); a.tau = tau;
    err = bf16 ? launch_mode<true, kExpBwdKV>(a, stream, "expect_bwd_kv_kernel")
               : launch_mode<false, kExpBwdKV>(a, stream, "expect_bwd_kv_kernel");
    if (err != hipSuccess) return err;
    // queries fixed, keys streamed: dQ
    ExpArgs b{};
    b.xr = q; b.ar = dy; b.xc = k; b.bc = v; b.yc = k; b.out2 = dq;
    b.bh = bh; b.n_r = static_cast<int>(n_q); b.n_c = static_cast<int>(n_k); b.tau = tau;
    return bf16 ? launch_mode<true, kExpBwdQ>(b, stream, "expect_bwd_q_kernel")
                : launch_mode<false, kExpBwdQ>(b, stream, "expect_bwd_q_kernel");
}

}  // namespace yoso
