// Sign-random-projection hash on MFMA (gfx950).
//
// Sec. 3.2 overview ("we sample a hash function f") with the hyperplane hash of
// the Fig. 2 caption: tau random hyperplanes per hash, concatenated sign bits.
// For every row x and column c = h*tau + t of R the projection P = x . R[:, c]
// is one entry of the dense product X R ([rows, 64] x [64, m*tau]); the code of
// hash h collects the tau signs of its columns, bit t = [P > 0].
//
// The product runs on v_mfma_f32_16x16x32_f16.  Each fp32 operand is split into
// an fp16 pair (hi + lo, ~21 significant bits, both truncated) and the three
// products hi*hi, hi*lo, lo*hi are accumulated in fp32, so a projection is off by
// at most about 2^-20 |x| |R[:, c]|.  Each row is first scaled by the power of two
// 2^(13 - e), max |x_i| < 2^e, so that its entries lie below 2^13 and their hi and
// lo parts are normal fp16 numbers whatever the row's magnitude (a positive scale
// changes no sign).  A bf16 row so scaled is exact as its hi parts (8 significant
// bits, within fp16's normal range down to 2^-27 of its largest entry), so bf16
// inputs take two products, hi*hi and hi*lo of R.
//
// Work split: a workgroup of 8 or 16 waves (two or one per CU, as LDS allows)
// converts R once into fp16 MFMA B-fragments in LDS and then walks tiles of 32
// rows per wave (persistent when there are more tiles than resident
// workgroups); each wave owns 32 rows of a tile (two 16-row MFMA tiles, so every
// B-fragment read from LDS feeds two row tiles; 16 rows when the tiles would not
// fill the resident workgroups) and all ceil(m*tau/16) column tiles.  The rows of a wave's next tile are loaded into registers while the
// current one is computed; the first tile's loads are issued before the
// conversion of R.  Signs are gathered with wave ballots: the four 64-bit
// ballots of a 16 x 16 output tile hold the 16-column sign segments of its 16
// rows, and they go to the wave's own LDS area unchanged (stored by lane 0).
// The same wave then cuts each hash's tau-bit field out of one or two segments
// and stores the codes of a row as consecutive uint16 values ([bh][n][m]
// layout).  Nothing in the tile loop waits for another wave.
#include "common.h"
#include "launch.h"
#include "timing.h"

namespace yoso {

namespace {

// 16-row MFMA tiles per wave and tile: RT = 2 (32 rows) where the workgroups fill
// the GPU, RT = 1 (16 rows, each wave's chain of products half as long) where they
// do not (one head of 512 rows: 15 -> 10 us; 384 x 512 rows: 33 -> 32 us with 2)
constexpr int kHashMaxRT = 2;

// fp32 -> fp16 (hi, lo) pairs, truncating (v_cvt_pkrtz_f16_f32 converts two values
// per instruction): hi = rtz(s), lo = rtz(s - hi), with s - hi exact in fp32;
// hi + lo keeps about 21 significant bits of s.
__device__ __forceinline__ void split8_rtz(const float v[8], float scale, half8 &hi, half8 &lo) {
#pragma unroll
    for (int p = 0; p < 4; p++) {
        const float a = v[2 * p] * scale, b = v[2 * p + 1] * scale;
        const auto h = __builtin_amdgcn_cvt_pkrtz(a, b);
        const auto l = __builtin_amdgcn_cvt_pkrtz(a - static_cast<float>(h[0]), b - static_cast<float>(h[1]));
        hi[2 * p] = static_cast<_Float16>(h[0]);
        hi[2 * p + 1] = static_cast<_Float16>(h[1]);
        lo[2 * p] = static_cast<_Float16>(l[0]);
        lo[2 * p + 1] = static_cast<_Float16>(l[1]);
    }
}

// Lane L feeds the A operand of row 16t + (L & 15), elements kb*32 + (L >> 4)*8 + [0, 8).
// Rows past the end load the last row (a valid address); their codes are not stored.
template <bool BF16, int RT>
__device__ __forceinline__ void hash_load_rows(const void *__restrict__ x, int64_t rows, int64_t base, int lane,
                                               float (&v)[RT][2][8]) {
#pragma unroll
    for (int t = 0; t < RT; t++) {
        int64_t row = base + 16 * t + (lane & 15);
        row = row < rows ? row : rows - 1;
#pragma unroll
        for (int kb = 0; kb < 2; kb++) load8<BF16>(x, row * D + kb * 32 + (lane >> 4) * 8, v[t][kb]);
    }
}

template <bool BF16, int WAVES, int RT>
__global__ __launch_bounds__(64 * WAVES) void hash_kernel(const void *__restrict__ x, int64_t rows,
                                                            const float *__restrict__ R, int m, int tau,
                                                            uint16_t *__restrict__ codes, int64_t num_tiles) {
    constexpr int kHashThreads = 64 * WAVES;
    constexpr int kHashWaveRows = 16 * RT;  // rows per wave and tile
    constexpr int kHashRowsPerTile = WAVES * kHashWaveRows;
    extern __shared__ __align__(16) unsigned char smem[];
    const int N = m * tau;               // columns of R
    const int NT = ((N + 31) >> 5) * 2;   // 16-column tiles, rounded up to a pair (extra columns are zero)
    half8 *frag = reinterpret_cast<half8 *>(smem);  // [NT][2 kb][2 hi/lo][64 lanes]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // the wave's ballots: [RT t][NT nt][4 i] uint64; bits [16g, 16g+16) of
    // ballot (t, nt, i) are the signs of row 16t + 4g + i, columns 16nt .. 16nt+15
    uint32_t *bal = reinterpret_cast<uint32_t *>(smem + (size_t)NT * 4096) + wave * RT * NT * 8;
    const uint16_t *seg = reinterpret_cast<const uint16_t *>(bal);

    // R -> fp16 B-fragments.  Fragment (nt, kb) lane L holds rows
    // k = kb*32 + (L>>4)*8 + [0,8) of column nt*16 + (L&15).  Four fragments per
    // thread at a time, all 32 loads issued before the first conversion.  The
    // loads of the first pass go out before the rows of the first tile, so the
    // conversion (and the barrier after it) waits for R only, and each wave
    // starts computing as soon as its own rows have arrived.
    float r[4][8];
    auto load_r = [&](int s0) {
#pragma unroll
        for (int u = 0; u < 4; u++) {
            const int s = s0 + u * kHashThreads;
            const int nt = s >> 7, kb = (s >> 6) & 1, L = s & 63;
            const int col = nt * 16 + (L & 15);
            const int k0 = kb * 32 + (L >> 4) * 8;
            // a clamped column keeps every address valid (k0 + i < 64 always);
            // values of columns past N are zeroed at conversion
            const float *src = R + (int64_t)k0 * N + (col < N ? col : N - 1);
#pragma unroll
            for (int i = 0; i < 8; i++) r[u][i] = src[(int64_t)i * N];
        }
    };
    load_r(tid);

    float xv[RT][2][8];
    int64_t tile = blockIdx.x;
    if (tile < num_tiles) hash_load_rows<BF16, RT>(x, rows, tile * kHashRowsPerTile + wave * kHashWaveRows, lane, xv);

    for (int s0 = tid; s0 < NT * 128; s0 += 4 * kHashThreads) {
        if (s0 != tid) load_r(s0);
#pragma unroll
        for (int u = 0; u < 4; u++) {
            const int s = s0 + u * kHashThreads;
            if (s >= NT * 128) break;
            const int nt = s >> 7, kb = (s >> 6) & 1, L = s & 63;
            const int col = nt * 16 + (L & 15);
            float v[8];
#pragma unroll
            for (int i = 0; i < 8; i++) v[i] = col < N ? r[u][i] : 0.f;
            half8 hi, lo;
            split8_rtz(v, 1.0f, hi, lo);
            frag[((nt * 2 + kb) * 2 + 0) * 64 + L] = hi;
            frag[((nt * 2 + kb) * 2 + 1) * 64 + L] = lo;
        }
    }
    __syncthreads();

    // Code cut: 64 / m rows per pass, lane -> (row offset cut_r, hash cut_h).
    const int rpp = 64 / m;
    const int cut_r = lane / m;
    const int cut_h = lane - cut_r * m;
    const bool cut_on = cut_r < rpp;
    const uint32_t mask = (1u << tau) - 1u;
    const int c0 = cut_h * tau, nt0 = c0 >> 4, sh = c0 & 15;
    const bool two_segs = sh + tau > 16;

    for (; tile < num_tiles; tile += gridDim.x) {
        const int64_t base = tile * kHashRowsPerTile + wave * kHashWaveRows;
        half8 ah[RT][2], al[RT][2];
#pragma unroll
        for (int t = 0; t < RT; t++) {
            // the row's largest |entry| (its 64 entries sit in the lanes L, L ^ 16,
            // L ^ 32, L ^ 48), then the power of two that brings it below 2^13
            float mx = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; kb++)
#pragma unroll
                for (int i = 0; i < 8; i++) mx = fmaxf(mx, fabsf(xv[t][kb][i]));
            mx = fmaxf(mx, __shfl_xor(mx, 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            // (max |x_i| = f 2^e, f in [0.5, 1); the scale stays a normal fp32 number
            // for every finite row, at most 2^126)
            int e = 0;
            if (mx > 0.f) frexpf(mx, &e);
            const float sc = ldexpf(1.0f, min(13 - e, 126));
#pragma unroll
            for (int kb = 0; kb < 2; kb++) split8_rtz(xv[t][kb], sc, ah[t][kb], al[t][kb]);
        }
        const int64_t next = tile + gridDim.x;
        if (next < num_tiles)
            hash_load_rows<BF16, RT>(x, rows, next * kHashRowsPerTile + wave * kHashWaveRows, lane, xv);

        for (int g0 = 0; g0 < NT; g0 += 2) {
            floatx4 acc[2][RT];
#pragma unroll
            for (int j = 0; j < 2; j++) {
                const int nt = g0 + j;
#pragma unroll
                for (int t = 0; t < RT; t++) acc[j][t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kb = 0; kb < 2; kb++) {
                    const half8 bh = frag[((nt * 2 + kb) * 2 + 0) * 64 + lane];
                    const half8 bl = frag[((nt * 2 + kb) * 2 + 1) * 64 + lane];
#pragma unroll
                    for (int t = 0; t < RT; t++) {
                        if constexpr (BF16) {
                            // (the lo parts of a scaled bf16 row are zero)
                            acc[j][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[t][kb], bh, acc[j][t], 0, 0, 0);
                            acc[j][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[t][kb], bl, acc[j][t], 0, 0, 0);
                        } else {
                            acc[j][t] = mfma3_16x16x32(ah[t][kb], al[t][kb], bh, bl, acc[j][t]);
                        }
                    }
                }
            }
            // acc[j][t][i] of lane L is P[row 16t + 4*(L>>4) + i][col (g0+j)*16 + (L&15)].
            // Ballot i collects, in bits [16g, 16g+16), the 16 column signs of row 16t + 4g + i.
            // The ballots are wave-uniform; lane 0 stores them.
            uint64_t b[RT][2][4];
#pragma unroll
            for (int t = 0; t < RT; t++)
#pragma unroll
                for (int j = 0; j < 2; j++)
#pragma unroll
                    for (int i = 0; i < 4; i++) b[t][j][i] = __ballot(acc[j][t][i] > 0.f);
            if (lane == 0) {
#pragma unroll
                for (int t = 0; t < RT; t++) {
#pragma unroll
                    for (int j = 0; j < 2; j++) {
                        uint4 *dst = reinterpret_cast<uint4 *>(bal + (t * NT + g0 + j) * 8);
                        dst[0] = make_uint4(static_cast<uint32_t>(b[t][j][0]), static_cast<uint32_t>(b[t][j][0] >> 32),
                                            static_cast<uint32_t>(b[t][j][1]), static_cast<uint32_t>(b[t][j][1] >> 32));
                        dst[1] = make_uint4(static_cast<uint32_t>(b[t][j][2]), static_cast<uint32_t>(b[t][j][2] >> 32),
                                            static_cast<uint32_t>(b[t][j][3]), static_cast<uint32_t>(b[t][j][3] >> 32));
                    }
                }
            }
        }

        // The wave's 32 rows are complete in its own ballots (LDS operations of one
        // wave are performed in order): cut the tau-bit fields and store the codes,
        // four passes at a time with their LDS reads issued first.
        // Segment (row 16t + 4g + i, column tile nt) is uint16 number
        // ((t*NT + nt)*4 + i)*4 + g; the next column tile is 16 further on.
        for (int r0 = 0; r0 < kHashWaveRows; r0 += 4 * rpp) {
            uint32_t v[4];
#pragma unroll
            for (int u = 0; u < 4; u++) {
                int r = r0 + u * rpp + cut_r;
                r = r < kHashWaveRows ? r : kHashWaveRows - 1;  // a valid address; not stored
                const int idx = (((r >> 4) * NT + nt0) * 4 + (r & 3)) * 4 + ((r >> 2) & 3);
                v[u] = static_cast<uint32_t>(seg[idx]) >> sh;
                if (two_segs) v[u] |= static_cast<uint32_t>(seg[idx + 16]) << (16 - sh);
            }
#pragma unroll
            for (int u = 0; u < 4; u++) {
                const int r = r0 + u * rpp + cut_r;
                const int64_t grow = base + r;
                if (cut_on && r < kHashWaveRows && grow < rows)
                    codes[grow * m + cut_h] = static_cast<uint16_t>(v[u] & mask);
            }
        }
    }
}

}  // namespace

// Launch shape of the hash kernel: 8-wave workgroups, two per CU, while two fit
// in the 160 KB of LDS of a CU; else one 16-wave workgroup per CU; else (the
// largest m*tau) one 8-wave workgroup per CU.
struct HashShape {
    int waves;
    int per_cu;
    size_t lds;
};

HashShape hash_shape(int m, int tau) {
    const int NT = ((m * tau + 31) >> 5) * 2;  // as in the kernel: column tiles rounded up to a pair
    const size_t frag = (size_t)NT * 4096, bal = (size_t)kHashMaxRT * NT * 32;
    if (frag + 8 * bal <= 80 * 1024) return {8, 2, frag + 8 * bal};
    if (frag + 16 * bal <= 156 * 1024) return {16, 1, frag + 16 * bal};
    return {8, 1, frag + 8 * bal};
}

size_t hash_lds_bytes(int m, int tau) { return hash_shape(m, tau).lds; }

hipError_t launch_hash(const void *x, bool bf16, int64_t bh, int64_t n, const float *R, int m, int tau,
                       uint16_t *codes, hipStream_t stream) {
    const int64_t rows = bh * n;
    if (rows == 0) return hipSuccess;
    const HashShape shape = hash_shape(m, tau);
    const int waves = shape.waves;
    const size_t lds = shape.lds;
    // Persistent workgroups, as many as are resident at once: each converts R
    // once, and with several tiles per workgroup the register prefetch overlaps
    // the loads of one tile with the work on another.
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) {
        (void)hipGetLastError();  // a failed query only changes the grid size
        cus = 256;
    }
    const int64_t resident = static_cast<int64_t>(cus) * shape.per_cu;
    // 32-row wave tiles where they fill the resident workgroups, else 16-row ones
    const int64_t tiles2 = (rows + waves * 32 - 1) / (waves * 32);
    const int rt = tiles2 < resident ? 1 : 2;
    const int64_t tiles = rt == 2 ? tiles2 : (rows + waves * 16 - 1) / (waves * 16);
    const int64_t grid = tiles < resident ? tiles : resident;
    KernelTimer timer("hash_kernel", stream);
    auto launch = [&](auto kernel, int threads) {
        hipLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(threads), lds, stream, x, rows, R, m, tau, codes, tiles);
    };
    if (bf16) {
        if (waves == 8) rt == 2 ? launch(hash_kernel<true, 8, 2>, 512) : launch(hash_kernel<true, 8, 1>, 512);
        else rt == 2 ? launch(hash_kernel<true, 16, 2>, 1024) : launch(hash_kernel<true, 16, 1>, 1024);
    } else {
        if (waves == 8) rt == 2 ? launch(hash_kernel<false, 8, 2>, 512) : launch(hash_kernel<false, 8, 1>, 512);
        else rt == 2 ? launch(hash_kernel<false, 16, 2>, 1024) : launch(hash_kernel<false, 16, 1>, 1024);
    }
    return hipGetLastError();
}

}  // namespace yoso
