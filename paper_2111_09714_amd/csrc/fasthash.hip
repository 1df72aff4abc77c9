// The fast hash (gfx950): Sec. 3.2, "Speed-up" -- the approximate random
// projection of Andoni et al. (2015).  Each rotation r = 0 .. ceil(m*tau/64) - 1 is
// the pseudo-random rotation H D3 H D2 H D1 (H the 64 x 64 Walsh-Hadamard matrix
// in Sylvester order, D_i diagonal +-1 from the caller's sign masks), and bit t of
// hash h is the sign of coordinate l of rotation r applied to the row, where
// h*tau + t = 64 r + l.  (The 1/64 scale that makes each row of the rotation as
// long as a Gaussian column changes no sign and is left out.)
//
// fast_hash_kernel applies the rotations row by row, as the paper does: one row
// per lane, its 64 values in registers, three rounds of "negate by D_i, then the
// six butterfly stages of H" per rotation -- d log2 d additions per round instead
// of the d^2 multiply-adds of a dense projection.  The work is fp32 VALU
// arithmetic (about 1.3k instructions per row and rotation), so the kernel is
// bound by the vector ALUs, not by HBM.
//
// The negations by D_i are sign-bit flips (one bitwise instruction per value).
// Folding them into the butterflies instead -- fused multiply-adds by a
// wave-uniform +-1 per pair of groups -- saves those instructions but needs about
// three scalar instructions per sign pair, and measured slower here.  The sign
// bits of a rotation are turned into codes at once, while they are still in
// registers: a hash whose tau columns straddle two rotations carries its low bits
// over to the next one.
//
// fast_hyperplanes_kernel writes the same rotations out as an explicit hyperplane
// matrix R (column 64 r + l of R = row l of rotation r, scaled by 1/64), so that
// the dense hash kernel reproduces the fast hash: one wave per 16 columns of R,
// lane l holding coordinate l of all 16, butterflies across lanes (the 16 columns
// interleaved so that their shuffles overlap).  All values are integers of
// magnitude at most 4096 before the final exact division by 64.
#include "common.h"
#include "launch.h"
#include "timing.h"

namespace yoso {

namespace {

constexpr int kFastThreads = 256;

// One round on the 64 values of a row held by this lane: negate the coordinates
// whose bit is set in the wave-uniform mask s, then the six butterfly stages of
// the Walsh-Hadamard transform (Sylvester order, unnormalised).
__device__ __forceinline__ void fast_round(float (&u)[64], uint64_t s) {
#pragma unroll
    for (int l = 0; l < 64; l++)
        u[l] = __uint_as_float(__float_as_uint(u[l]) ^ (static_cast<uint32_t>((s >> l) & 1u) << 31));
#pragma unroll
    for (int h = 1; h < 64; h <<= 1) {
#pragma unroll
        for (int l = 0; l < 64; l++) {
            if (l & h) continue;
            const float a = u[l], b = u[l + h];
            u[l] = a + b;
            u[l + h] = a - b;
        }
    }
}

// TAU > 0 (a divisor of 64, known at compile time): every rotation holds exactly
// 64 / TAU whole hashes, and each sign bit is ORed straight into its code at a
// fixed position.  TAU == 0: any tau (the run-time argument); the sign bits of a
// rotation go into one 64-bit word from which the hashes are cut, a hash that
// straddles two rotations carrying its low bits over.  One row per lane.
template <bool BF16, int TAU>
__global__ __launch_bounds__(kFastThreads) void fast_hash_kernel(const void *__restrict__ x, int64_t rows,
                                                                 const uint64_t *__restrict__ signs, int m, int tau_arg,
                                                                 uint16_t *__restrict__ codes) {
    const int tau = TAU > 0 ? TAU : tau_arg;
    const int ncol = m * tau;
    const int nrot = (ncol + 63) >> 6;
    const uint32_t mask = (1u << tau) - 1u;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * kFastThreads + threadIdx.x;
    // rows past the end (in a wave that holds valid rows) hash the last row; not stored
    const int64_t src = row < rows ? row : rows - 1;
    const bool store = row < rows;
    uint16_t *dst = codes + (store ? row : 0) * m;
    float v[64];
#pragma unroll
    for (int c = 0; c < 64; c += 8) load8<BF16>(x, src * D + c, v + c);

    uint32_t cur = 0;   // TAU == 0: bits gathered so far of the hash in progress
    uint32_t held = 0;  // TAU == 0: a finished even-numbered code waiting for its odd partner
    int h = 0;          // TAU == 0: hash in progress (wave-uniform)
    for (int r = 0; r < nrot; r++) {
        float u[64];
#pragma unroll
        for (int l = 0; l < 64; l++) u[l] = v[l];
#pragma unroll
        for (int round = 0; round < 3; round++) fast_round(u, signs[3 * r + round]);
        // the sign test is strict: a zero gives bit 0
        if constexpr (TAU > 0) {
            constexpr int HPR = 64 / TAU;  // hashes per rotation
            uint32_t code[HPR];
#pragma unroll
            for (int j = 0; j < HPR; j++) code[j] = 0;
#pragma unroll
            for (int l = 0; l < 64; l++) code[l / TAU] |= (u[l] > 0.f ? 1u : 0u) << (l % TAU);
            const int h0 = r * HPR;
            if (store) {
                if (HPR % 2 == 0 && (m & 1) == 0) {
#pragma unroll
                    for (int j = 0; j < HPR; j += 2)
                        if (h0 + j < m) reinterpret_cast<uint32_t *>(dst)[(h0 + j) >> 1] = code[j] | (code[j + 1] << 16);
                } else {
#pragma unroll
                    for (int j = 0; j < HPR; j++)
                        if (h0 + j < m) dst[h0 + j] = static_cast<uint16_t>(code[j]);
                }
            }
        } else {
            uint32_t w0 = 0, w1 = 0;
#pragma unroll
            for (int l = 0; l < 32; l++) {
                w0 |= (u[l] > 0.f ? 1u : 0u) << l;
                w1 |= (u[l + 32] > 0.f ? 1u : 0u) << l;
            }
            const uint64_t W = (static_cast<uint64_t>(w1) << 32) | w0;  // bit l: column 64 r + l
            const int c_lo = 64 * r, c_hi = ncol < c_lo + 64 ? ncol : c_lo + 64;
            // hashes with columns in [c_lo, c_hi): the first may have begun in the
            // previous rotation, the last may end in the next one
            for (; h * tau < c_hi; h++) {
                const int c0 = h * tau;
                cur |= c0 >= c_lo ? static_cast<uint32_t>(W >> (c0 - c_lo)) : static_cast<uint32_t>(W << (c_lo - c0));
                if (c0 + tau > c_hi) break;  // continues in the next rotation
                const uint32_t code = cur & mask;
                cur = 0;
                if (m & 1) {
                    if (store) dst[h] = static_cast<uint16_t>(code);
                } else if (h & 1) {
                    if (store) reinterpret_cast<uint32_t *>(dst)[h >> 1] = held | (code << 16);
                } else {
                    held = code;
                }
            }
        }
    }
}

// Explicit hyperplanes of the rotations: workgroup (r, q) computes columns
// j = 16q .. 16q+15 of H D3 H D2 H D1 (lane l = row l), i.e. entry j of every row
// of rotation r, and stores them scaled by 1/64 as row j of R's columns 64r + l.
__global__ __launch_bounds__(64) void fast_hyperplanes_kernel(const uint64_t *__restrict__ signs, int ncol,
                                                              float *__restrict__ R) {
    const int r = blockIdx.x >> 2, q = blockIdx.x & 3;
    const int lane = threadIdx.x;
    float v[16];
#pragma unroll
    for (int c = 0; c < 16; c++) v[c] = lane == 16 * q + c ? 1.f : 0.f;
#pragma unroll
    for (int round = 0; round < 3; round++) {
        const bool neg = (signs[3 * r + round] >> lane) & 1u;
#pragma unroll
        for (int c = 0; c < 16; c++) v[c] = neg ? -v[c] : v[c];
#pragma unroll
        for (int h = 1; h < 64; h <<= 1) {
            float p[16];
#pragma unroll
            for (int c = 0; c < 16; c++) p[c] = __shfl_xor(v[c], h);
#pragma unroll
            for (int c = 0; c < 16; c++) v[c] = (lane & h) ? p[c] - v[c] : v[c] + p[c];
        }
    }
    const int col = r * 64 + lane;
    if (col < ncol) {
#pragma unroll
        for (int c = 0; c < 16; c++) R[(int64_t)(16 * q + c) * ncol + col] = v[c] * (1.f / 64.f);
    }
}

}  // namespace

hipError_t launch_fast_hash(const void *x, bool bf16, int64_t bh, int64_t n, const uint64_t *signs, int m, int tau,
                            uint16_t *codes, hipStream_t stream) {
    const int64_t rows = bh * n;
    if (rows == 0) return hipSuccess;
    const int64_t blocks = (rows + kFastThreads - 1) / kFastThreads;  // rows < 2^40: fits the grid
    const dim3 grid(static_cast<unsigned>(blocks)), block(kFastThreads);
    KernelTimer timer("fast_hash_kernel", stream);
    auto go = [&](auto kernel) {
        hipLaunchKernelGGL(kernel, grid, block, 0, stream, x, rows, signs, m, tau, codes);
    };
    switch (tau) {
        case 1: bf16 ? go(fast_hash_kernel<true, 1>) : go(fast_hash_kernel<false, 1>); break;
        case 2: bf16 ? go(fast_hash_kernel<true, 2>) : go(fast_hash_kernel<false, 2>); break;
        case 4: bf16 ? go(fast_hash_kernel<true, 4>) : go(fast_hash_kernel<false, 4>); break;
        case 8: bf16 ? go(fast_hash_kernel<true, 8>) : go(fast_hash_kernel<false, 8>); break;
        default: bf16 ? go(fast_hash_kernel<true, 0>) : go(fast_hash_kernel<false, 0>); break;
    }
    return hipGetLastError();
}

hipError_t launch_fast_hyperplanes(const uint64_t *signs, int m, int tau, float *R, hipStream_t stream) {
    const int ncol = m * tau;
    const int nrot = (ncol + 63) / 64;
    KernelTimer timer("fast_hyperplanes_kernel", stream);
    hipLaunchKernelGGL(fast_hyperplanes_kernel, dim3(4 * nrot), dim3(64), 0, stream, signs, ncol, R);
    return hipGetLastError();
}

}  // namespace yoso
