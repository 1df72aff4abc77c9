// Sign-random-projection hash on MFMA (gfx950).
//
// Sec. 3.2 overview ("we sample a hash function f") with the hyperplane hash of
// the Fig. 2 caption: tau random hyperplanes per hash, concatenated sign bits.
// For every row x and column c = h*tau + t of R the projection P = x . R[:, c]
// is one entry of the dense product X R ([rows, 64] x [64, m*tau]); the code of
// hash h collects the tau signs of its columns, bit t = [P > 0].
//
// The product runs on v_mfma_f32_16x16x32_f16.  Each fp32 operand is split into
// an fp16 pair (hi + lo, ~22 significant bits) and the three products hi*hi,
// hi*lo, lo*hi are accumulated in fp32, which reproduces the fp32 dot product to
// about 1e-6 (rows are scaled by 2^8 first so that lo parts of unit-vector
// entries stay normal fp16 numbers; the scaling does not change any sign).
//
// Work split: a workgroup (4 waves) owns 64-row tiles; each wave owns 16 rows
// and all ceil(m*tau/16) column tiles.  R is converted once per workgroup into
// fp16 MFMA B-fragments in LDS.  Signs are gathered with wave ballots into a
// per-row bit vector in LDS, from which each hash's tau-bit field is cut and
// stored as uint16 in the [bh][n][m] layout (the m codes of a row are
// contiguous).
#include "common.h"
#include "launch.h"
#include "timing.h"

namespace yoso {

namespace {

constexpr int kHashRowsPerTile = 64;
constexpr int kHashGroup = 8;  // column tiles accumulated at once (8 x floatx4)

template <bool BF16>
__global__ __launch_bounds__(256) void hash_kernel(const void *__restrict__ x, int64_t rows,
                                                   const float *__restrict__ R, int m, int tau,
                                                   uint16_t *__restrict__ codes, int64_t num_tiles) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int N = m * tau;               // columns of R
    const int NT = (N + 15) >> 4;         // 16-column tiles
    const int NW = (NT + 1) >> 1;         // 32-bit words of sign bits per row
    const int NWP = NW | 1;               // padded row stride (odd: fewer bank conflicts)
    half8 *frag = reinterpret_cast<half8 *>(smem);                        // [NT][2 kb][2 hi/lo][64 lanes]
    uint32_t *bits = reinterpret_cast<uint32_t *>(smem + (size_t)NT * 4096);  // [64 rows][NWP]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    // R -> fp16 B-fragments.  Fragment (nt, kb) lane L holds rows
    // k = kb*32 + (L>>4)*8 + [0,8) of column nt*16 + (L&15).  Four fragments per
    // thread at a time, all 32 loads issued before the first conversion (the
    // conversion is latency-bound, and it is repeated by every workgroup).
    for (int s0 = tid; s0 < NT * 128; s0 += 4 * 256) {
        float r[4][8];
#pragma unroll
        for (int u = 0; u < 4; u++) {
            const int s = s0 + u * 256;
            const int nt = s >> 7, kb = (s >> 6) & 1, L = s & 63;
            const int col = nt * 16 + (L & 15);
            const int k0 = kb * 32 + (L >> 4) * 8;
            const bool ok = s < NT * 128 && col < N;
            // (a clamped, always valid address; out-of-range values are zeroed below)
            const float *src = R + (ok ? (int64_t)k0 * N + col : 0);
#pragma unroll
            for (int i = 0; i < 8; i++) r[u][i] = src[ok ? (int64_t)i * N : 0];
        }
#pragma unroll
        for (int u = 0; u < 4; u++) {
            const int s = s0 + u * 256;
            if (s >= NT * 128) break;
            const int nt = s >> 7, kb = (s >> 6) & 1, L = s & 63;
            const int col = nt * 16 + (L & 15);
            float v[8];
#pragma unroll
            for (int i = 0; i < 8; i++) v[i] = col < N ? r[u][i] : 0.f;
            half8 hi, lo;
            split8(v, 1.0f, hi, lo);
            frag[((nt * 2 + kb) * 2 + 0) * 64 + L] = hi;
            frag[((nt * 2 + kb) * 2 + 1) * 64 + L] = lo;
        }
    }
    __syncthreads();

    const int kq = lane >> 4;       // which 8-element k chunk this lane feeds
    const int rsub = lane & 15;     // row within the wave's 16 rows
    for (int64_t tile = blockIdx.x; tile < num_tiles; tile += gridDim.x) {
        const int64_t row = tile * kHashRowsPerTile + wave * 16 + rsub;
        half8 ah[2], al[2];
#pragma unroll
        for (int kb = 0; kb < 2; kb++) {
            float v[8];
            if (row < rows) {
                load8<BF16>(x, row * D + kb * 32 + kq * 8, v);
            } else {
#pragma unroll
                for (int i = 0; i < 8; i++) v[i] = 0.f;
            }
            split8(v, 256.0f, ah[kb], al[kb]);
        }

        for (int g0 = 0; g0 < NT; g0 += kHashGroup) {
            floatx4 acc[kHashGroup];
#pragma unroll
            for (int j = 0; j < kHashGroup; j++) {
                acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
                const int nt = g0 + j;
                if (nt < NT) {
#pragma unroll
                    for (int kb = 0; kb < 2; kb++) {
                        const half8 bh = frag[((nt * 2 + kb) * 2 + 0) * 64 + lane];
                        const half8 bl = frag[((nt * 2 + kb) * 2 + 1) * 64 + lane];
                        acc[j] = mfma3_16x16x32(ah[kb], al[kb], bh, bl, acc[j]);
                    }
                }
            }
            // acc[j][i] of lane L is P[row 4*(L>>4)+i][col (g0+j)*16 + (L&15)].
            // Ballot i collects, in bits [16g, 16g+16), the 16 column signs of row 4g+i.
#pragma unroll
            for (int j = 0; j < kHashGroup; j += 2) {
                uint32_t word = 0;
#pragma unroll
                for (int half = 0; half < 2; half++) {
                    const int nt = g0 + j + half;
                    if (nt < NT) {
                        const uint64_t b0 = __ballot(acc[j + half][0] > 0.f);
                        const uint64_t b1 = __ballot(acc[j + half][1] > 0.f);
                        const uint64_t b2 = __ballot(acc[j + half][2] > 0.f);
                        const uint64_t b3 = __ballot(acc[j + half][3] > 0.f);
                        // lane rsub stands for row rsub = 4g + i of this wave
                        const int i = rsub & 3, g = rsub >> 2;
                        const uint64_t b = (i == 0) ? b0 : (i == 1) ? b1 : (i == 2) ? b2 : b3;
                        word |= static_cast<uint32_t>((b >> (16 * g)) & 0xFFFFu) << (16 * half);
                    }
                }
                const int w = (g0 + j) >> 1;
                if (lane < 16 && w < NW) bits[(wave * 16 + lane) * NWP + w] = word;
            }
        }
        __syncthreads();

        // Cut the tau-bit field of every (row, hash) out of the row's bit vector;
        // consecutive threads write consecutive hashes of a row.
        const uint32_t mask = (1u << tau) - 1u;
        for (int p = tid; p < kHashRowsPerTile * m; p += 256) {
            const int r = p / m, h = p - r * m;
            const int64_t grow = tile * kHashRowsPerTile + r;
            if (grow < rows) {
                const int o = h * tau, w = o >> 5, s = o & 31;
                uint32_t v = bits[r * NWP + w] >> s;
                if (s + tau > 32) v |= bits[r * NWP + w + 1] << (32 - s);
                codes[grow * m + h] = static_cast<uint16_t>(v & mask);
            }
        }
        __syncthreads();
    }
}

// Hyperplanes of the fast hash (Sec. 3.2 "Speed-up": the approximate random
// projection of Andoni et al. 2015, a pseudo-random rotation H D3 H D2 H D1 with H
// the 64 x 64 Walsh-Hadamard matrix and D_i random +-1 diagonals).  On gfx950 the
// rotation is not applied row by row: at d = 64 its 3 * 64 * 6 butterfly additions
// per 64 projections cost more VALU time than the dense product costs on MFMA.  So
// each rotation is expanded once into the 64 rows it projects onto, and the hash
// kernel above evaluates them like any hyperplane matrix R.
//
// Thread j of workgroup r pushes e_j through the three rounds (negate the
// coordinates that D_i flips, then the in-place Walsh-Hadamard butterflies in
// natural order), which yields column j of H D3 H D2 H D1, i.e. entry j of each of
// the rotation's 64 rows; scaled by 1/64 they are row j of R's columns 64r .. 64r+63.
// Every intermediate is an integer of magnitude at most 4096, so the fp32 result
// is exact (each entry a multiple of 1/64 of magnitude at most 8).
__global__ __launch_bounds__(64) void fast_hyperplanes_kernel(const uint64_t *__restrict__ signs, int ncol,
                                                              float *__restrict__ R) {
    const int r = blockIdx.x;
    const int j = threadIdx.x;
    float v[64];
#pragma unroll
    for (int l = 0; l < 64; l++) v[l] = l == j ? 1.f : 0.f;
#pragma unroll
    for (int round = 0; round < 3; round++) {
        const uint64_t s = signs[3 * r + round];
#pragma unroll
        for (int l = 0; l < 64; l++) v[l] = ((s >> l) & 1u) ? -v[l] : v[l];
#pragma unroll
        for (int h = 1; h < 64; h <<= 1) {
#pragma unroll
            for (int l = 0; l < 64; l++) {
                if (l & h) continue;
                const float a = v[l], b = v[l + h];
                v[l] = a + b;
                v[l + h] = a - b;
            }
        }
    }
    float *dst = R + (int64_t)j * ncol + r * 64;
    const int valid = ncol - r * 64;  // columns of this rotation that R holds (the last one may be cut)
#pragma unroll
    for (int l = 0; l < 64; l++)
        if (l < valid) dst[l] = v[l] * (1.f / 64.f);
}

}  // namespace

size_t hash_lds_bytes(int m, int tau) {
    const int N = m * tau;
    const int NT = (N + 15) >> 4;
    const int NW = (NT + 1) >> 1;
    return (size_t)NT * 4096 + (size_t)kHashRowsPerTile * (NW | 1) * 4;
}

hipError_t launch_hash(const void *x, bool bf16, int64_t bh, int64_t n, const float *R, int m, int tau,
                       uint16_t *codes, hipStream_t stream) {
    const int64_t rows = bh * n;
    if (rows == 0) return hipSuccess;
    const int64_t tiles = (rows + kHashRowsPerTile - 1) / kHashRowsPerTile;
    // persistent workgroups (two per CU): each converts R once for several tiles
    const int64_t grid = tiles < 512 ? tiles : 512;
    const size_t lds = hash_lds_bytes(m, tau);
    KernelTimer timer("hash_kernel", stream);
    if (bf16) {
        hipLaunchKernelGGL(hash_kernel<true>, dim3((unsigned)grid), dim3(256), lds, stream, x, rows, R, m, tau,
                           codes, tiles);
    } else {
        hipLaunchKernelGGL(hash_kernel<false>, dim3((unsigned)grid), dim3(256), lds, stream, x, rows, R, m, tau,
                           codes, tiles);
    }
    return hipGetLastError();
}

hipError_t launch_fast_hyperplanes(const uint64_t *signs, int m, int tau, float *R, hipStream_t stream) {
    const int ncol = m * tau;
    const int nrot = (ncol + 63) / 64;
    KernelTimer timer("fast_hyperplanes_kernel", stream);
    hipLaunchKernelGGL(fast_hyperplanes_kernel, dim3(nrot), dim3(64), 0, stream, signs, ncol, R);
    return hipGetLastError();
}

}  // namespace yoso
