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
//   codes_t_kernel long sequences: the codes transposed to [bh][m][n], so that the
//                  sort reads each (head, hash) column contiguously.
//   sort_kernel    one workgroup per (head, hash, side): histogram of the codes,
//                  exclusive scan -> bucket offsets, then the rows in bucket order
//                  as packed entries (code << 16 | row): a stable counting sort in
//                  LDS (rows of a bucket in increasing index), so the order in which
//                  the pair passes accumulate, and hence every result, is reproducible.
//   absmax_kernel  partial maxima of |Q|, |dY|, |K|, |V| per head, from which every
//                  consumer derives the same power-of-two scale per (head, tensor).
//   split_kernel   Q, K, V, dY -> fp16 (hi, lo) rows, each head's tensor scaled by
//                  2^(13 - e) with max|x| < 2^e, so that hi and lo stay normal fp16
//                  numbers whatever the data's magnitude (bf16 inputs: hi only).
//   pass_kernel    one workgroup per (head, hash, side).  Each wave walks 16-row
//                  tiles of sorted rows; the partners that can collide with a tile
//                  form one contiguous range of sorted partners, visited 16 at a
//                  time:  S^T = A'_y A_x^T (16x16x32 MFMA), masked by code equality,
//                  out^T += B_y^T S^T (16x16x16 MFMA).  The partner rows of the next
//                  sub-tile are fetched while the current one computes; B_y is
//                  transposed through a per-wave LDS tile.  The finished tile is the
//                  hash's share of out for those rows; it is stored, not added, into a
//                  partial buffer (each row of each hash is written exactly once, so no
//                  atomics are needed) as a fixed-point row with one power-of-two
//                  exponent: 24 bits per value (16 high, 8 low), or 16 bits for bf16
//                  outputs.  With *YOSO's weights (STAR) it runs over the m tau
//                  derived hashes of drop_bit_kernel.
//   bucket_kernel  the buckets large enough for the table form: per bucket and side
//                  M = sum_y a'_y b_y^T (64 x 64), then out_x = s a_x^T M for its rows,
//                  stored as the same partial rows (the pass kernel skips them).
//   reduce_kernel  out[b][x] = sum over the m hashes of the partial rows, in hash
//                  order (deterministic), written as fp32 or bf16.
//   dense_kernel   short sequences: C = sum_h B_h from the sorted bucket lists, then
//                  dQ, dK and dV as dense masked MFMA blocks, no partial rows.
//   dense_fwd_kernel  the forward for many heads of short sequences, Y = (1/m) C V,
//                  C counted from bit planes of the codes.
// gfx950's global fp32 atomics sustain roughly 1.3 TB/s of payload, so a plain
// store of every partial plus one coalesced reduction beats accumulating with
// atomics.  Every fp32 product uses three fp16 MFMAs (hi*hi + hi*lo + lo*hi).
// Before S is split for the second product it is scaled per row by 2^-(2 + e_x),
// ||a_x|| < 2^e_x, which keeps |S| below 2^14 (||a'_y|| < 2^16 after the head
// scaling) and keeps a small row's S as precise as a large one's; the row's
// factor is undone when its partial row is stored.
#include "common.h"
#include "launch.h"
#include "timing.h"

namespace yoso {

namespace {

// Sort workgroups: four waves when the column or the entries are staged in LDS;
// eight when neither is (long sequences: more rows per workgroup to place, 89 ->
// 72 us at n = 32768) and tau <= 10 (the larger tables and masks of tau 11-12 do not
// fit twice); one for short sequences over many heads (below).
constexpr int kSortThreads = 256;
constexpr int kSortThreadsWide = 512;
// Short sequences over many heads: one wave per (head, hash, side).  The work of a
// workgroup is then a few 64-row steps and its fixed cost (zeroing, scan, barriers)
// is paid by one wave, with many more workgroups resident per CU (384 x 512: 90 ->
// 56 us; at 4096 rows four waves are faster, and a single head gains nothing).
constexpr int kSortThreadsNarrow = 64;
constexpr int64_t kSortNarrowN = 1024;
constexpr int64_t kSortNarrowBlocks = 2048;

// Waves of a sort workgroup that place rows: each needs a 64-bit lane mask per bucket.
__host__ __device__ constexpr int sort_placing_waves(int tau, int waves) { return tau <= 10 ? waves : 1; }

// Dynamic LDS of a sort workgroup of `nt` threads before staging: per-wave counts,
// scan scratch, placing waves' masks.
inline size_t sort_base_lds(int nt, int tau) {
    return (static_cast<size_t>(nt / 64) * (size_t{1} << tau) + nt) * 4 +
           static_cast<size_t>(sort_placing_waves(tau, nt / 64)) * (size_t{1} << tau) * 8;
}
constexpr size_t kSortStageLds = 120 * 1024;  // LDS bound of a sort workgroup that stages codes and entries
constexpr size_t kSortEntLds = 160 * 1024;    // LDS bound of a sort workgroup that stages its entries only
constexpr int kPassThreads = 256;
constexpr int kPassWaves = kPassThreads / 64;
constexpr int kReduceThreads = 256;
constexpr int kTileBytes = 16 * 512;   // LDS bytes of one wave's operand tile
constexpr int kPlanTiles = 256;        // row tiles planned per run (multiple of kPassThreads)
constexpr int kExpLds = 16384;         // rows whose exponents a pass block stages in LDS
constexpr int kEntPad = 16;            // at least this many sentinel entries after each unit's sorted entries
constexpr int kMaxParts = 8;           // partial maxima per (head, tensor)
constexpr int kMantBytes = 16 * 128;   // LDS bytes of a finished tile's 16-bit mantissas (the low bytes follow)

// Entries per unit: n rounded up to a multiple of 4 (16-byte aligned units), then
// at least kEntPad sentinels.
__host__ __device__ constexpr int64_t ent_stride(int64_t n) { return ((n + 3) & ~int64_t{3}) + kEntPad; }
constexpr uint32_t kSentinel = 0xFFFF0000u;  // code 0xFFFF (no real code), row 0
// A pass block's copy of a row entry whose bucket takes the table form gets this
// code: no partner matches it and its partial row is not stored.
constexpr uint32_t kSkipCode = 0xFFFEu;

// ---- the table form of a large bucket
// For bucket c of one hash, with b_q queries and b_k keys, the pairs cost 4 d b_q b_k
// multiply-adds (S and the output, both sides).  The same sums follow from one d x d
// matrix per side: M_c = sum_y a'_y b_y^T over the partners, then out_x = s a_x^T M_c
// for every row, 2 d^2 (b_q + b_k) multiply-adds (the table subroutine of Sec. 3.3
// restricted to one bucket).  The table form wins when b_q b_k > (d / 2)(b_q + b_k)
// counted in multiply-adds; its dense 64 x 64 products run the matrix cores far
// better than the masked 16 x 16 pair tiles, so the bucket switches over at a
// threshold below d / 2.  kTableT >= 16 keeps every table bucket above 16 rows on
// both sides, so within a 16-row tile its rows are a prefix and/or a suffix.
constexpr int kTableT = 24;
static_assert(kTableT >= 16, "table buckets must span more than one row tile");

__device__ __forceinline__ bool table_bucket(int32_t bq, int32_t bk, int t) {
    return t > 0 && static_cast<int64_t>(bq) * bk > static_cast<int64_t>(t) * (bq + bk);
}

// ---------------------------------------------------------------- counting sort
// Codes transposed to [bh][m][n] (codes_t_kernel): one block's column is contiguous.
// (Read from the [bh][n][m] layout, every 2-byte code of a column was a 64-byte
// segment of its own, and each of a head's m hash blocks fetched the whole array.)
// VEC (m a multiple of 8): the tile's rows are read 8 codes (16 bytes) at a time;
// its columns are written 8 codes at a time where the 8 rows are all there.
template <bool VEC>
__global__ __launch_bounds__(256) void codes_t_kernel(const uint16_t *__restrict__ in, uint16_t *__restrict__ out,
                                                      int64_t bh, int64_t n, int m) {
    // item (b, row tile of 64, column tile of 64), grid-stride; the tile is padded so
    // that the transposed reads of a row of it hit distinct banks
    __shared__ uint16_t tile[64][66];
    const int64_t ntr = (n + 63) / 64;
    const int ntc = (m + 63) / 64;
    for (int64_t blk = blockIdx.x; blk < bh * ntr * ntc; blk += gridDim.x) {
        const int tc = static_cast<int>(blk % ntc);
        const int64_t tr = (blk / ntc) % ntr;
        const int64_t b = blk / (static_cast<int64_t>(ntc) * ntr);
        const int64_t r0 = tr * 64;
        const int c0 = tc * 64;
        if constexpr (VEC) {
            // 64 rows x 8 groups of 8 codes: one 16-byte load per thread and pass
            for (int e = threadIdx.x; e < 64 * 8; e += 256) {
                const int r = e >> 3, c8 = (e & 7) * 8;
                if (r0 + r < n && c0 + c8 < m) {
                    const uint4 w = *reinterpret_cast<const uint4 *>(in + (b * n + r0 + r) * m + c0 + c8);
                    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                    for (int i = 0; i < 4; i++) {
                        tile[c8 + 2 * i][r] = static_cast<uint16_t>(ws[i]);
                        tile[c8 + 2 * i + 1][r] = static_cast<uint16_t>(ws[i] >> 16);
                    }
                }
            }
        } else {
            for (int e = threadIdx.x; e < 64 * 64; e += 256) {
                const int r = e >> 6, c = e & 63;
                if (r0 + r < n && c0 + c < m) tile[c][r] = in[(b * n + r0 + r) * m + c0 + c];
            }
        }
        __syncthreads();
        for (int e = threadIdx.x; e < 64 * 8; e += 256) {
            const int c = e >> 3, r8 = (e & 7) * 8;
            if (c0 + c >= m) continue;
            uint16_t *dst = out + (b * m + c0 + c) * n + r0 + r8;
            if (VEC && r0 + r8 + 8 <= n && ((reinterpret_cast<uintptr_t>(dst) & 15) == 0)) {
                uint4 w;
                w.x = tile[c][r8] | (static_cast<uint32_t>(tile[c][r8 + 1]) << 16);
                w.y = tile[c][r8 + 2] | (static_cast<uint32_t>(tile[c][r8 + 3]) << 16);
                w.z = tile[c][r8 + 4] | (static_cast<uint32_t>(tile[c][r8 + 5]) << 16);
                w.w = tile[c][r8 + 6] | (static_cast<uint32_t>(tile[c][r8 + 7]) << 16);
                *reinterpret_cast<uint4 *>(dst) = w;
            } else {
                for (int i = 0; i < 8 && r0 + r8 + i < n; i++) dst[i] = tile[c][r8 + i];
            }
        }
        __syncthreads();  // the tile is refilled for the next item of the stride
    }
}

// unit = b*m + h reads column h of head b: with stride m from the codes as given
// ([bh][n][m], `transposed` false), or contiguous from codes_t_kernel's copy.
template <int NT>
__global__ __launch_bounds__(NT) void sort_kernel(const uint16_t *__restrict__ qcodes,
                                                            const uint16_t *__restrict__ kcodes, int m,
                                                            int64_t n_q, int64_t n_k, int tau, bool transposed,
                                                            bool stage_codes, bool stage_ent,
                                                            int32_t *__restrict__ qoff, int32_t *__restrict__ koff,
                                                            uint32_t *__restrict__ qent,
                                                            uint32_t *__restrict__ kent) {
    // [NW][buckets] per-wave counts, then per-wave cursors; + [NT]
    // scan scratch; + [placing waves][buckets] 64-bit lane masks; when `stage_ent`,
    // the sorted entries, which are then written out whole (single scattered 4-byte
    // stores would each cost a partial-line write); when `stage_codes`, the column's
    // codes (read from memory once)
    constexpr int NW = NT / 64;
    extern __shared__ int32_t hist[];
    const int B = 1 << tau;
    int32_t *scan = hist + NW * B;
    const int pw = sort_placing_waves(tau, NW);
    unsigned long long *masks = reinterpret_cast<unsigned long long *>(scan + NT);
    uint32_t *est = reinterpret_cast<uint32_t *>(masks + pw * B);
    const int64_t unit = blockIdx.x >> 1;
    const bool kside = blockIdx.x & 1;
    const int64_t b = unit / m;
    const int h = static_cast<int>(unit - b * m);
    const int64_t n = kside ? n_k : n_q;
    uint16_t *cst = reinterpret_cast<uint16_t *>(est + (stage_ent ? n : 0));
    const uint16_t *codes = (kside ? kcodes : qcodes) + (transposed ? (b * m + h) * n : b * n * m + h);
    const int64_t cstride = transposed ? 1 : m;
    int32_t *off = (kside ? koff : qoff) + unit * (B + 1);
    uint32_t *ent = (kside ? kent : qent) + unit * ent_stride(n);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // placing wave w owns the contiguous rows [r0, r1); the order is then rows in
    // increasing index within each bucket, independent of any timing
    const int64_t seg = (n + pw - 1) / pw;
    const int64_t r0 = wave < pw ? min(n, wave * seg) : n, r1 = wave < pw ? min(n, r0 + seg) : n;

    for (int c = tid; c < NW * B; c += NT) hist[c] = 0;
    for (int c = tid; c < pw * B; c += NT) masks[c] = 0ull;
    __syncthreads();
    {
        // sixteen codes per lane in flight before their counts are added (one at a
        // time, every load's latency was paid in turn); rows past r1 read row r1 - 1
        // and are not counted
        constexpr int U = 16;
        for (int64_t i0 = r0 + lane; i0 < r1; i0 += 64 * U) {
            uint32_t cc[U];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int64_t i = i0 + 64 * u;
                cc[u] = codes[(i < r1 ? i : r1 - 1) * cstride];
            }
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int64_t i = i0 + 64 * u;
                if (i < r1) {
                    const int c = static_cast<int>(cc[u]) & (B - 1);
                    if (stage_codes) cst[i] = static_cast<uint16_t>(c);
                    atomicAdd(&hist[wave * B + c], 1);
                }
            }
        }
    }
    __syncthreads();

    // bucket offsets (exclusive scan of the totals; thread t owns buckets
    // [t*per, (t+1)*per)), and each wave's first position in each bucket
    const int per = (B + NT - 1) / NT;
    const int c0 = tid * per;
    int32_t local = 0;
    for (int c = c0; c < c0 + per && c < B; c++)
        for (int w = 0; w < NW; w++) local += hist[w * B + c];
    // (inclusive scan: within each wave by shuffles, then the totals of the waves
    // before it)
    int32_t incl = local;
#pragma unroll
    for (int s = 1; s < 64; s <<= 1) {
        const int32_t v = __shfl_up(incl, s);
        if (lane >= s) incl += v;
    }
    if (lane == 63) scan[wave] = incl;
    __syncthreads();
    for (int w = 0; w < wave; w++) incl += scan[w];
    int32_t run = incl - local;
    for (int c = c0; c < c0 + per && c < B; c++) {
        off[c] = run;
        for (int w = 0; w < NW; w++) {
            const int32_t k = hist[w * B + c];
            hist[w * B + c] = run;  // becomes wave w's cursor in bucket c
            run += k;
        }
    }
    if (tid == 0) off[B] = static_cast<int32_t>(n);
    __syncthreads();

    // each placing wave places its rows 64 at a time, in order.  Every lane sets its
    // bit in its bucket's lane mask; the mask then gives the lane its rank among the
    // lanes of its bucket (bits below its own) and the bucket's count; the lowest
    // such lane advances the cursor and clears the mask.  (The mask and cursor
    // arrays are private to the wave and LDS executes one wave's accesses in order.)
    if (wave < pw) {
        int32_t *cur = hist + wave * B;
        unsigned long long *mk = masks + wave * B;
        for (int64_t base = r0; base < r1; base += 64) {
            const int64_t i = base + lane;
            const bool valid = i < r1;
            const int64_t ic = valid ? i : r1 - 1;
            const uint32_t c = stage_codes ? cst[ic] : codes[ic * cstride] & (B - 1);
            if (valid) atomicOr(&mk[c], 1ull << lane);
            const unsigned long long mask = mk[c];
            const int32_t first = cur[c];
            const int rank = __popcll(mask & ((1ull << lane) - 1ull));
            if (valid) {
                const uint32_t e = (c << 16) | static_cast<uint32_t>(i);
                if (stage_ent)
                    est[first + rank] = e;
                else
                    ent[first + rank] = e;
                if (rank == 0) {
                    cur[c] = first + __popcll(mask);
                    mk[c] = 0ull;
                }
            }
        }
    }
    if (stage_ent) {
        __syncthreads();
        // the entries, then the sentinels, 16 bytes per thread (ent_stride is a
        // multiple of 4 and the unit's entry array starts 16-byte aligned)
        const int64_t n4 = n >> 2;
        for (int64_t e = tid; e < ent_stride(n) / 4; e += NT) {
            uint4 w;
            if (e < n4) {
                w = reinterpret_cast<const uint4 *>(est)[e];
            } else {
                const int64_t j = 4 * e;
                w.x = j < n ? est[j] : kSentinel;
                w.y = j + 1 < n ? est[j + 1] : kSentinel;
                w.z = j + 2 < n ? est[j + 2] : kSentinel;
                w.w = j + 3 < n ? est[j + 3] : kSentinel;
            }
            reinterpret_cast<uint4 *>(ent)[e] = w;
        }
    } else {
        for (int64_t i = n + tid; i < ent_stride(n); i += NT) ent[i] = kSentinel;
    }
}

// ---------------------------------------------------------------- per-head scales
// Tensor t of head b: 0 = Q, 1 = dY (n_q rows), 2 = K, 3 = V (n_k rows).
// Block (b*4 + t)*kMaxParts + p takes the p-th of kMaxParts contiguous row ranges
// and writes max |x| over it; pmax[(b*4 + t)*kMaxParts + p].
template <bool BF16>
__global__ __launch_bounds__(256) void absmax_kernel(const void *__restrict__ q, const void *__restrict__ dy,
                                                     const void *__restrict__ k, const void *__restrict__ v,
                                                     int64_t n_q, int64_t n_k, float *__restrict__ pmax) {
    __shared__ float wred[4];
    const int64_t blk = blockIdx.x;
    const int p = static_cast<int>(blk % kMaxParts);
    const int64_t bt = blk / kMaxParts;
    const int t = static_cast<int>(bt & 3);
    const int64_t b = bt >> 2;
    const void *src = t == 0 ? q : t == 1 ? dy : t == 2 ? k : v;
    const int64_t n = t < 2 ? n_q : n_k;
    const int64_t per = (n + kMaxParts - 1) / kMaxParts;
    const int64_t r0 = min(n, p * per), r1 = min(n, r0 + per);
    const int64_t base = (b * n + r0) * D, count = (r1 - r0) * D;
    float mx = 0.f;
    constexpr int U = 4;  // loads in flight per thread
    for (int64_t e0 = static_cast<int64_t>(threadIdx.x) * 8; e0 < count; e0 += 256 * 8 * U) {
        float x[U][8];
#pragma unroll
        for (int u = 0; u < U; u++) {
            const int64_t e = e0 + u * 256 * 8;
            load8<BF16>(src, base + (e < count ? e : 0), x[u]);
        }
#pragma unroll
        for (int u = 0; u < U; u++) {
            if (e0 + u * 256 * 8 < count) {
#pragma unroll
                for (int i = 0; i < 8; i++) mx = fmaxf(mx, fabsf(x[u][i]));
            }
        }
    }
    mx = wave_max(mx);
    if ((threadIdx.x & 63) == 0) wred[threadIdx.x >> 6] = mx;
    __syncthreads();
    if (threadIdx.x == 0) pmax[blk] = fmaxf(fmaxf(wred[0], wred[1]), fmaxf(wred[2], wred[3]));
}

// e with max |x| < 2^e over tensor t of head b (the tensor is scaled by 2^(13 - e)).
__device__ __forceinline__ int head_exp(const float *pmax, int64_t b, int t) {
    const float4 *p = reinterpret_cast<const float4 *>(pmax + (b * 4 + t) * kMaxParts);
    const float4 x = p[0], y = p[1];
    const float m = fmaxf(fmaxf(fmaxf(x.x, x.y), fmaxf(x.z, x.w)), fmaxf(fmaxf(y.x, y.y), fmaxf(y.z, y.w)));
    return pow2_above(m);
}

// ---------------------------------------------------------------- pair passes
struct Side {
    const uint32_t *ent;  // [units][ent_stride(n)]: (code << 16 | row) in bucket order, then sentinels
    const int32_t *off;   // [units][2^tau + 1] bucket offsets
    int64_t n;
};

struct PassArgs {
    Side q, k;
    // Q, K, V, dY split into fp16 (hi, lo) pairs by split_kernel: row r holds 64 hi
    // halves then 64 lo halves, each head's tensor scaled by its power of two
    const _Float16 *qs, *ks, *vs, *dys;
    const float *pmax;               // per-head partial maxima (absmax_kernel)
    int16_t *pq, *pk;                // partials [bh][n][m][64]: high 16 bits of the 24-bit mantissas
    uint8_t *lq, *lk;                // [bh][n][m][64]: their low 8 bits
    int8_t *eq, *ek;                 // their exponents [bh][m][n] (one block writes one n-byte run)
    // per row of dY (the dQ side's rows) and of V (the dK side's): e with ||a|| < 2^e
    // for the fp16 pairs above [bh][n] (split_kernel)
    const int8_t *rexq, *rexk;
    int64_t bh;
    int m, tau;
    float scale;                     // tau / (2m)
    int tab_t;                       // table form for buckets with b_q b_k > tab_t (b_q + b_k); 0: none
    bool p16;                        // 16-bit partial rows carrying their exponents (bf16 outputs)
};

// ---- the wave's LDS tile
// Operands reach the MFMA layouts through one 8 KiB LDS tile per wave.  Global
// loads are coalesced: the 16 lanes of a quarter-wave read 256 contiguous bytes
// of one row (where an MFMA-layout load would touch 16 rows per quarter-wave and
// make 4x as many cache requests).  16-byte chunks are XOR-swizzled within a row
// so that the MFMA-layout reads (16 rows, one chunk each), the transpose reads
// (4 or 8 rows x 32 bytes) and the row writes all hit distinct banks.
//   partner tile: 16 rows x 512 B  [a' hi | a' lo | b hi | b lo], 128 B each
//   row tile:     16 rows x 256 B  [a hi | a lo]
//   out tile:     16 rows x 256 B  (64 fp32)
__device__ __forceinline__ uint32_t swz(int row, int chunk, int row_bytes) {
    // f permutes 0..15; f(r) mod 8 differs within every aligned group of 8 rows and
    // f(r) >> 1 differs within every aligned group of 8 (so also of 4) rows
    const int f = ((2 * row + ((row >> 2) & 1)) & 15) ^ ((row >> 3) & 1);
    return static_cast<uint32_t>(row * row_bytes + ((chunk ^ f) << 4));
}

template <typename T>
__device__ __forceinline__ T lds_ld(const unsigned char *base, uint32_t off) {
    return *reinterpret_cast<const T *>(base + off);
}
template <typename T>
__device__ __forceinline__ void lds_st(unsigned char *base, uint32_t off, const T &v) {
    *reinterpret_cast<T *>(base + off) = v;
}

// HI1 (bf16 inputs): a bf16 value scaled by a power of two is an fp16 number
// wherever it lies in fp16's normal range (every value above 2^-27 of its head's
// largest), so the lo halves of the fp16 (hi, lo) copies are zero.  Only the hi
// halves are then loaded, staged and multiplied: slot i of lane (q, cl) holds hi
// chunk cl & 7 of partner (or row) 4q + 2i + (cl >> 3), two slots per lane; in the
// general form slot i holds chunk cl of partner (or row) 4q + i, four slots.
template <bool HI1>
__device__ __forceinline__ int slot_row(int q, int cl, int i) { return HI1 ? 4 * q + 2 * i + (cl >> 3) : 4 * q + i; }
template <bool HI1>
__device__ __forceinline__ int slot_chunk(int cl) { return HI1 ? (cl & 7) : cl; }
// the entry of slot i from the lane's entries of partners (rows) 4q .. 4q+3
template <bool HI1>
__device__ __forceinline__ uint32_t slot_entry(const uint4 &e4, int cl, int i) {
    const uint32_t e[4] = {e4.x, e4.y, e4.z, e4.w};
    if constexpr (HI1) return (cl >> 3) ? e[2 * i + 1] : e[2 * i];
    return e[i];
}

// One 16-partner sub-tile as loaded: slot i of a' (a[i]) and of b (b[i]).
struct Sub {
    uint4 a[4], b[4];
};

// `pe` holds this lane's entries of partners 4q .. 4q+3 (code << 16 | row), one
// aligned 16-byte load.  Entries past the unit's end are sentinels (row 0, an
// impossible code), so every load is in bounds and a partner outside the tile's
// buckets is masked by its code.
template <bool HI1>
__device__ __forceinline__ void load_sub(Sub &s, const uint4 &pe, const _Float16 *apar, const _Float16 *bpar,
                                         int cl) {
#pragma unroll
    for (int i = 0; i < (HI1 ? 2 : 4); i++) {
        const uint32_t off = (slot_entry<HI1>(pe, cl, i) & 0xFFFFu) * (4 * D) + 16 * slot_chunk<HI1>(cl);
        s.a[i] = ld<uint4>(apar, off);
        s.b[i] = ld<uint4>(bpar, off);
    }
}

// The 16 rows of a tile as loaded (slots as above); `re4` holds the entries of rows
// 4q .. 4q+3.
template <bool HI1>
__device__ __forceinline__ void load_row_tile(uint4 r[4], const uint4 &re4, const _Float16 *arow, int cl) {
#pragma unroll
    for (int i = 0; i < (HI1 ? 2 : 4); i++)
        r[i] = ld<uint4>(arow, (slot_entry<HI1>(re4, cl, i) & 0xFFFFu) * (4 * D) + 16 * slot_chunk<HI1>(cl));
}

// Rows through the tile into the MFMA B-operand layout of S^T: lane (g, c) gets
// row c, dims kb*32 + 8g + [0, 8) (hi and lo; HI1: hi, and lo is zero).
template <bool HI1>
__device__ __forceinline__ void stage_rows(const uint4 r[4], unsigned char *tile, int q, int cl, int g, int c,
                                          half8 rh[2], half8 rl[2]) {
#pragma unroll
    for (int i = 0; i < (HI1 ? 2 : 4); i++) lds_st(tile, swz(slot_row<HI1>(q, cl, i), slot_chunk<HI1>(cl), 256), r[i]);
#pragma unroll
    for (int kb = 0; kb < 2; kb++) {
        rh[kb] = lds_ld<half8>(tile, swz(c, kb * 4 + g, 256));
        if constexpr (HI1)
            rl[kb] = half8{};
        else
            rl[kb] = lds_ld<half8>(tile, swz(c, 8 + kb * 4 + g, 256));
    }
}

// The rows' own b vectors (the q of a query row, the k of a key row; used by
// *YOSO for q.k) through the second half of the tile into the same B-operand
// layout: lane (g, c) gets row c, dims kb*32 + 8g + [0, 8).
template <bool HI1>
__device__ __forceinline__ void stage_rows_b(const uint4 r[4], unsigned char *tile, int q, int cl, int g, int c,
                                             half8 bh[2], half8 bl[2]) {
    unsigned char *t = tile + 16 * 256;
#pragma unroll
    for (int i = 0; i < (HI1 ? 2 : 4); i++) lds_st(t, swz(slot_row<HI1>(q, cl, i), slot_chunk<HI1>(cl), 256), r[i]);
#pragma unroll
    for (int kb = 0; kb < 2; kb++) {
        bh[kb] = lds_ld<half8>(t, swz(c, kb * 4 + g, 256));
        if constexpr (HI1)
            bl[kb] = half8{};
        else
            bl[kb] = lds_ld<half8>(t, swz(c, 8 + kb * 4 + g, 256));
    }
}

__device__ __forceinline__ half4 tr_load(const unsigned char *p) {
    typedef short short4v __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) short4v lds_short4;
    return __builtin_bit_cast(half4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4 *)(p)));
}

// Sub-tile into the tile (LDS executes one wave's accesses in order, so the reads
// of compute_sub see these writes; the tile is private to the wave).
template <bool HI1>
__device__ __forceinline__ void publish_sub(const Sub &s, unsigned char *tile, int q, int cl) {
#pragma unroll
    for (int i = 0; i < (HI1 ? 2 : 4); i++) {
        lds_st(tile, swz(slot_row<HI1>(q, cl, i), slot_chunk<HI1>(cl), 512), s.a[i]);
        lds_st(tile, swz(slot_row<HI1>(q, cl, i), 16 + slot_chunk<HI1>(cl), 512), s.b[i]);
    }
}

// out^T += B_y^T S^T for the sub-tile in the tile: S^T = A'_y A_x^T masked by
// code equality.  `pe` as in load_sub: in the MFMA layout it holds the entries of
// exactly the partners 4g+i whose S^T values this lane computes.
// *YOSO's weight bound: 1 - x^2 is raised to at least 1/64 (|x| <= 0.99216).
constexpr float kStarFloor = 1.0f / 64.0f;

// HI1: the lo halves are zero; only the products with a hi operand on both sides of
// a' . a and b . S remain (S itself is a general fp32 value and keeps its pair).
template <bool STAR, bool HI1>
__device__ __forceinline__ void compute_sub(const unsigned char *tile, const uint4 &pe, const half8 rh[2],
                                            const half8 rl[2], const half8 rbh[2], const half8 rbl[2], float xscale,
                                            int rcode, float sfac, int g, int c, floatx4 outT[4]) {
    // A'_y in the A-operand layout: lane (g, c) = partner c, dims kb*32 + 8g + [0, 8)
    half8 ah[2], al[2];
#pragma unroll
    for (int kb = 0; kb < 2; kb++) {
        ah[kb] = lds_ld<half8>(tile, swz(c, kb * 4 + g, 512));
        if constexpr (!HI1) al[kb] = lds_ld<half8>(tile, swz(c, 8 + kb * 4 + g, 512));
    }
    // B_y^T as the A operand of a 16x16x16 MFMA: lane (g, c) needs partners 4g+i of
    // dim 16dt+c.  ds_read_b64_tr_b16 gives destination lane 4a+b of a 16-lane
    // group element b of the 8 bytes addressed by source lanes 4i+a (i = 0..3), so
    // source lane 4i+a addresses partner 4g+i, dims 16dt + 4a .. +3 (chunk 2dt +
    // a/2 of the b hi or lo part, half a%2 of it).
    const int pr = 4 * g + (c >> 2), a4 = c & 3;
    half4 bth[4], btl[4];
#pragma unroll
    for (int dt = 0; dt < 4; dt++) {
        bth[dt] = tr_load(tile + swz(pr, 16 + 2 * dt + (a4 >> 1), 512) + 8 * (a4 & 1));
        if constexpr (!HI1) btl[dt] = tr_load(tile + swz(pr, 24 + 2 * dt + (a4 >> 1), 512) + 8 * (a4 & 1));
    }
    // S^T[partner 4g+i][row c]: two independent accumulation chains (one per 32
    // dims) interleaved, so consecutive MFMAs do not wait on each other
    const floatx4 z = {0.f, 0.f, 0.f, 0.f};
    floatx4 s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[0], rh[0], z, 0, 0, 0);
    floatx4 s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[1], rh[1], z, 0, 0, 0);
    if constexpr (!HI1) {
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[0], rl[0], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[1], rl[1], s1, 0, 0, 0);
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[0], rh[0], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[1], rh[1], s1, 0, 0, 0);
    }
    const floatx4 st = s0 + s1;
    const uint32_t e[4] = {pe.x, pe.y, pe.z, pe.w};
    float sv[4];
#pragma unroll
    for (int i = 0; i < 4; i++) sv[i] = static_cast<int>(e[i] >> 16) == rcode ? st[i] : 0.f;
    if constexpr (STAR) {
        // x = q.k of each pair (the partner's b from the tile in the A-operand
        // layout, the row's own b in the B layout), then the weight
        // 1 / (pi sqrt(max(1 - x^2, 1/64))) of eq. (gradient-q)
        half8 xh[2], xl[2];
#pragma unroll
        for (int kb = 0; kb < 2; kb++) {
            xh[kb] = lds_ld<half8>(tile, swz(c, 16 + kb * 4 + g, 512));
            if constexpr (!HI1) xl[kb] = lds_ld<half8>(tile, swz(c, 24 + kb * 4 + g, 512));
        }
        floatx4 x0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(xh[0], rbh[0], z, 0, 0, 0);
        floatx4 x1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(xh[1], rbh[1], z, 0, 0, 0);
        if constexpr (!HI1) {
            x0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(xh[0], rbl[0], x0, 0, 0, 0);
            x1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(xh[1], rbl[1], x1, 0, 0, 0);
            x0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(xl[0], rbh[0], x0, 0, 0, 0);
            x1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(xl[1], rbh[1], x1, 0, 0, 0);
        }
        const floatx4 xt = x0 + x1;
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const float x = xt[i] * xscale;
            sv[i] *= rsqrtf(fmaxf(fmaf(-x, x, 1.0f), kStarFloor)) * 0.31830988618379067f;
        }
    }
    // the row's factor 2^-(2 + e_c): |S| < 2^14 (see the header), hi and lo stay normal
    half4 sh, sl;
    if constexpr (STAR)
        split4(sv, sfac, sh, sl);  // sv carries the weight, a product of its own
    else
        split4_pow2(sv, sfac, sh, sl);
    // out^T += B_y^T S^T (hi*hi + hi*lo + lo*hi), the four dim blocks interleaved.
    // The general form takes hi*lo + lo*hi in one 16x16x32 product over the
    // concatenated operands [B hi | B lo] and [S lo ; S hi] (a contraction does not
    // depend on the order of its k index, only on both operands using the same one),
    // then hi*hi in a 16x16x16 product.
    if constexpr (HI1) {
#pragma unroll
        for (int dt = 0; dt < 4; dt++) outT[dt] = __builtin_amdgcn_mfma_f32_16x16x16f16(bth[dt], sh, outT[dt], 0, 0, 0);
#pragma unroll
        for (int dt = 0; dt < 4; dt++) outT[dt] = __builtin_amdgcn_mfma_f32_16x16x16f16(bth[dt], sl, outT[dt], 0, 0, 0);
    } else {
        const half8 slh = __builtin_shufflevector(sl, sh, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
        for (int dt = 0; dt < 4; dt++) {
            const half8 bt = __builtin_shufflevector(bth[dt], btl[dt], 0, 1, 2, 3, 4, 5, 6, 7);
            outT[dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(bt, slh, outT[dt], 0, 0, 0);
        }
#pragma unroll
        for (int dt = 0; dt < 4; dt++) outT[dt] = __builtin_amdgcn_mfma_f32_16x16x16f16(bth[dt], sh, outT[dt], 0, 0, 0);
    }
}

// Byte offset of 8-byte chunk ch (int16 dims 4ch .. 4ch+3) of the mantissa row in
// slot s of the tile (16 slots of 128 bytes).  Row r sits in slot r ^ ((r >> 2) & 1),
// so the two rows that a half-wave reads in the row-major pass have opposite slot
// parity (opposite halves of the 64 banks); within a slot the 16-byte unit of a
// chunk is XORed with s >> 1, so the eight same-parity rows that a half-wave writes
// from the MFMA layout (one unit each) hit distinct banks.
__device__ __forceinline__ int mant_slot(int r) { return r ^ ((r >> 2) & 1); }
__device__ __forceinline__ uint32_t mant_off(int s, int ch) {
    return static_cast<uint32_t>(s * 128 + (((ch >> 1) ^ (s >> 1)) << 4) + ((ch & 1) << 3));
}
// Byte offset of dword w (low bytes of dims 4w .. 4w+3) of row r's 64 low bytes,
// after the mantissas: row r = 4a + b sits in 64-byte slot 4a + ((a + b) & 3), and
// the dword's group of four (w >> 2) is XORed with a.  MFMA-layout writes (rows c,
// dwords 4dt + g) and row-major reads (rows 4q + i, dword cl: the rows whose high
// parts the lane stores, so that both stores of a row share its address) then both
// fall on 64 distinct banks.
__device__ __forceinline__ uint32_t low_off(int r, int w) {
    const int s = (r & 12) | ((r + (r >> 2)) & 3);
    return static_cast<uint32_t>(kMantBytes + s * 64 + ((((w >> 2) ^ (r >> 2)) & 3) << 4) + ((w & 3) << 2));
}

// Write the partial rows of a finished tile: lane (g, c) holds out[row c][16dt +
// 4g + (0..3)] / orow, orow being the lane's row factor.  A partial row is stored
// as 24-bit fixed point: one exponent e with max|value| < 2^e, and per value the
// integer M = round(value * 2^(22 - e)), |M| <= 2^22, kept in offset binary as
// U = M + 2^22 (0 <= U <= 2^23): its high 16 bits (U >> 8) and its low 8 bits
// (U & 255); value = (U - 2^22) 2^(e - 22) (rounding error at most 2^(e - 23),
// i.e. below 2^-22 of the row's largest value).  U comes from one fused
// multiply-add: value * 2^(22 - e) + 1.5 * 2^23 lies in (2^23, 2^24), where fp32
// numbers are the integers, so the sum rounded to nearest (ties to even, as M is
// rounded) is 1.5 * 2^23 + M, whose low 24 bits are U (2^24 itself, M = 2^22, has
// low bits 2^23 = U as well).  The row
// maximum and M are computed where the MFMA leaves the values (16 per lane, the
// rest of the row in the lanes 16, 32 and 48 away: two permlane swaps); both parts
// then go through the tile so that each quarter-wave stores one whole 128-byte
// high-part row and one whole 64-byte low-part row.  The stores are non-temporal:
// the partials are read once, by the reduction, and should not evict the operands
// from L2.  Exponents go to the block's LDS copy of its exponent row when it fits
// (written out whole at the end: single-byte stores scattered over the row would
// each cost a partial-line write), else straight to memory.  p16 (bf16 outputs):
// 16-bit rows that carry their own exponent (below).  Rows past nvalid and rows
// whose entry carries kSkipCode (their bucket takes the table form) are not stored.
// (P16 fixes p16 at compile time for the bf16 kernels; the pair kernels pass the
// constant for fp32 too, the table-form kernel the run-time value, false: each
// choice was measured faster for its kernel, by 3% and 4%)
template <bool P16>
__device__ __forceinline__ void store_tile(unsigned char *tile, int16_t *part, uint8_t *plow, int8_t *pexp,
                                           int8_t *ex_lds, bool ex_in_lds, int m, bool rt_p16,
                                           const uint32_t *tile_ent, int nvalid, int q, int cl, int g, int c,
                                           const floatx4 outT[4], float orow) {
    const bool p16 = P16 || rt_p16;
    // nothing to store when every row of the tile takes the table form (wave-uniform)
    if (__builtin_amdgcn_ballot_w64(c < nvalid && (tile_ent[c] >> 16) != kSkipCode) == 0) return;
    // max |value| of row c over this lane's 16 values (a chain of 3-input maxima),
    // then over the row's 4 lanes
    float mx = 0.f;
#pragma unroll
    for (int dt = 0; dt < 4; dt++) {
        mx = fmaxf(fmaxf(mx, fabsf(outT[dt][0])), fabsf(outT[dt][1]));
        mx = fmaxf(fmaxf(mx, fabsf(outT[dt][2])), fabsf(outT[dt][3]));
    }
    {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
        mx = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    }
    {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
        mx = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    }
    // e with max|value| < 2^e, from the biased exponent field of the scaled row
    // maximum (0 gives a tiny e whose mantissas are all 0), clamped to [-100, 127]
    // so that 2^(fb - e) and 2^(e - fb) stay normal floats (a row below 2^-100 only
    // keeps fewer bits; one whose largest value reaches 2^127, next to fp32's
    // overflow, is outside the format)
    const float mxs = mx * orow;
    const int e = min(max(static_cast<int>((__float_as_uint(mxs) >> 23) & 0xFFu) - 126, -100), 127);
    // value * 2^(fb - e) lies in (-2^fb, 2^fb): a power-of-two scaling of the
    // rounded product value * orow, so the row maximum stays below 2^fb before
    // rounding (and at most 2^fb after, hence the clamp of 16-bit values).  fb = 22
    // (24-bit rows), or 15 with p16 (16-bit rows: bf16 outputs, whose own rounding
    // is 2^-9)
    const int fb = p16 ? 15 : 22;
    const int mmax = (1 << fb) - 1;
    const float sc = mx > 0.f ? __uint_as_float(static_cast<uint32_t>(127 + fb - e) << 23) * orow : 0.f;
    if (!p16 && g == 0 && c < nvalid && (tile_ent[c] >> 16) != kSkipCode) {
        const uint32_t row = tile_ent[c] & 0xFFFFu;
        if (ex_in_lds) ex_lds[row] = static_cast<int8_t>(e);
        else pexp[row] = static_cast<int8_t>(e);
    }
    typedef unsigned int uint2v __attribute__((ext_vector_type(2)));
    const int sw = mant_slot(c);
#pragma unroll
    for (int dt = 0; dt < 4; dt++) {
        int mm[4];
        if (p16) {
#pragma unroll
            for (int j = 0; j < 4; j++) mm[j] = min(max(__float2int_rn(outT[dt][j] * sc), -mmax), mmax);
        } else {
#pragma unroll
            for (int j = 0; j < 4; j++) mm[j] = __float_as_int(fmaf(outT[dt][j], sc, 12582912.0f));  // 1.5 * 2^23
        }
        if (p16 && dt == 0 && g == 0) {
            // 16-bit rows carry their exponent in the record: the two low bits of
            // values 0 .. 3 (held by this lane) are bits 2j, 2j+1 of e, and those four
            // values keep 14 bits (2^-13 of the row's largest value); the row is then
            // one whole 128-byte line with nothing stored beside it
            const uint32_t eb = static_cast<uint32_t>(e) & 0xFFu;
#pragma unroll
            for (int j = 0; j < 4; j++)
                mm[j] = static_cast<int>(static_cast<uint32_t>(min(max(__float2int_rn(outT[0][j] * sc * 0.25f), -8191),
                                                                   8191))
                                         << 2) |
                        static_cast<int>((eb >> (2 * j)) & 3u);
        }
        // byte permutes: the high parts are bytes 1-2 of each U, the low part byte 0
        // (v_perm_b32 picks any bytes of a register pair: {first operand : second})
        const uint32_t u[4] = {static_cast<uint32_t>(mm[0]), static_cast<uint32_t>(mm[1]),
                               static_cast<uint32_t>(mm[2]), static_cast<uint32_t>(mm[3])};
        // (p16: the low 16 bits of each M)
        const uint32_t hsel = p16 ? 0x05040100u : 0x06050201u;
        uint2v w;
        w.x = __builtin_amdgcn_perm(u[1], u[0], hsel);
        w.y = __builtin_amdgcn_perm(u[3], u[2], hsel);
        lds_st(tile, mant_off(sw, 4 * dt + g), w);
        if (!p16) {
            const uint32_t lo01 = __builtin_amdgcn_perm(u[1], u[0], 0x0C0C0400u);  // [b0 of M0, b0 of M1, 0, 0]
            const uint32_t lo23 = __builtin_amdgcn_perm(u[3], u[2], 0x0C0C0400u);
            lds_st(tile, low_off(c, 4 * dt + g), __builtin_amdgcn_perm(lo23, lo01, 0x05040100u));
        }
    }
    // rows 4q + i: this lane's chunk cl of each high-part row, then the four stores
    uint2v w[4];
    uint32_t lw[4];
#pragma unroll
    for (int i = 0; i < 4; i++) w[i] = lds_ld<uint2v>(tile, mant_off(mant_slot(4 * q + i), cl));
    // rows 4q + i: dword cl of each low-part row
    if (!p16) {
#pragma unroll
        for (int i = 0; i < 4; i++) lw[i] = lds_ld<uint32_t>(tile, low_off(4 * q + i, cl));
    }
    const uint4 e4 = reinterpret_cast<const uint4 *>(tile_ent)[q];
    const uint32_t re[4] = {e4.x, e4.y, e4.z, e4.w};
    // (row, hash) record index row * m by a full-rate 24-bit multiply (row < 2^16,
    // m < 2^10), kept opaque so that it is not folded back into a 32-bit multiply
    // by m * 64
    auto rec = [&](uint32_t row) {
        uint32_t r = __umul24(row, static_cast<uint32_t>(m));
        asm("" : "+v"(r));
        return static_cast<uint64_t>(r);
    };
#pragma unroll
    for (int i = 0; i < 4; i++) {
        if (4 * q + i < nvalid && (re[i] >> 16) != kSkipCode) {
            const uint64_t rr = rec(re[i] & 0xFFFFu) * D;
            __builtin_nontemporal_store(w[i], reinterpret_cast<uint2v *>(part + rr) + cl);
            if (!p16) __builtin_nontemporal_store(lw[i], reinterpret_cast<uint32_t *>(plow + rr) + cl);
        }
    }
}

__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// STAR: *YOSO's estimator on derived codes (see launch_backward_star); its extra
// operands run at one workgroup per CU.
template <bool STAR, bool HI1>
__global__ __launch_bounds__(kPassThreads, STAR ? 1 : 2) void pass_kernel(PassArgs a) {
    __shared__ __align__(16) unsigned char tiles_lds[kPassWaves * kTileBytes];
    __shared__ int32_t plan_beg[kPlanTiles];      // first partner of each row tile's bucket range
    __shared__ int32_t plan_x[kPlanTiles + 1];    // exclusive prefix of the tiles' sub-tile counts
    __shared__ int32_t scan_tmp[kPassWaves];     // the waves' count totals
    __shared__ __align__(16) uint32_t row_ent[kPlanTiles * 16];  // the run's sorted row entries
    __shared__ __align__(16) int8_t ex_lds[kExpLds];               // the block's exponent row
    __shared__ uint8_t tab_lds[STAR ? 1 : 4096];  // 1 where the bucket takes the table form

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
    const int n_r = static_cast<int>(kside ? a.k.n : a.q.n);
    const int n_p = static_cast<int>(kside ? a.q.n : a.k.n);
    const uint32_t *rent = (kside ? a.k.ent : a.q.ent) + unit * ent_stride(n_r);
    const uint32_t *pent = (kside ? a.q.ent : a.k.ent) + unit * ent_stride(n_p);
    const int32_t *poff = (kside ? a.q.off : a.k.off) + unit * ((1 << a.tau) + 1);
    const _Float16 *arow = (kside ? a.vs : a.dys) + b * n_r * (2 * D);
    const _Float16 *apar = (kside ? a.dys : a.vs) + b * n_p * (2 * D);
    const _Float16 *bpar = (kside ? a.qs : a.ks) + b * n_p * (2 * D);
    const _Float16 *brow = (kside ? a.ks : a.qs) + b * n_r * (2 * D);  // *YOSO only
    const int8_t *rexp = (kside ? a.rexk : a.rexq) + b * n_r;         // ||a_r|| < 2^rexp[r]
    // *YOSO: x = (q 2^(13 - e_Q)) . (k 2^(13 - e_K)) * xscale
    const float xscale = STAR ? ldexpf(1.0f, head_exp(a.pmax, b, 0) + head_exp(a.pmax, b, 2) - 26) : 0.f;
    // partial row (row r, hash h) starts r*m*64 elements past these bases, its
    // exponent r bytes past the other
    int16_t *part = (kside ? a.pk : a.pq) + ((b * n_r) * a.m + h) * D;
    uint8_t *plow = (kside ? a.lk : a.lq) + ((b * n_r) * a.m + h) * D;
    int8_t *pexp = (kside ? a.ek : a.eq) + (b * a.m + h) * n_r;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = uni(tid >> 6);  // wave-uniform, so the scheduling below stays scalar
    const int g = lane >> 4, c = lane & 15;  // MFMA layout
    const int q = lane >> 4, cl = lane & 15; // coalesced layout: quarter q, 16-byte chunk cl
    unsigned char *tile = tiles_lds + wave * kTileBytes;
    const int tiles = (n_r + 15) >> 4;
    // the operands carry the head scales 2^(13 - e) of a (rows), a' (partners) and
    // b (partners), and S the row factor 2^-(2 + e_c): out = s * outT * 2^(e_a +
    // e_a' + e_b - 39) * 2^(2 + e_c)
    // (tensors: 0 Q, 1 dY, 2 K, 3 V; dQ: a = dY, a' = V, b = K; dK: a = V, a' = dY, b = Q)
    const int esum = head_exp(a.pmax, b, kside ? 3 : 1) + head_exp(a.pmax, b, kside ? 1 : 3) +
                     head_exp(a.pmax, b, kside ? 0 : 2);
    const float oscale = ldexpf(a.scale, esum - 39 + 2);
    const bool ex_in_lds = !HI1 && n_r <= kExpLds;  // (16-bit rows carry their exponents)

    // buckets in the table form (bucket_kernel writes their rows' partials): the
    // plan leaves their rows out of every tile's partner range and the run's copy
    // of their entries carries kSkipCode
    const int nb = 1 << a.tau;
    const bool tab = !STAR && a.tab_t > 0;
    const int32_t *roff = (kside ? a.k.off : a.q.off) + unit * (nb + 1);
    if (tab) {
        const int32_t *qo = a.q.off + unit * (nb + 1), *ko = a.k.off + unit * (nb + 1);
        for (int cb = tid; cb < nb; cb += kPassThreads)
            tab_lds[cb] = table_bucket(qo[cb + 1] - qo[cb], ko[cb + 1] - ko[cb], a.tab_t) ? 1 : 0;
        __syncthreads();
    }
    auto is_tab = [&](uint32_t code) { return tab && code < static_cast<uint32_t>(nb) && tab_lds[code]; };

    for (int T0 = 0; T0 < tiles; T0 += kPlanTiles) {
        const int nt = min(kPlanTiles, tiles - T0);
        // ---- plan: the bucket range of every row tile and its number of 16-partner sub-tiles
        {
            constexpr int PER = kPlanTiles / kPassThreads;
            int cnt[PER];
            int local = 0;
#pragma unroll
            for (int j = 0; j < PER; j++) {
                const int i = tid * PER + j;
                cnt[j] = 0;
                if (i < nt) {
                    const int r0 = (T0 + i) * 16;
                    int lo = r0, hi = r0 + min(16, n_r - r0);  // the tile's rows that take pairs
                    uint32_t cf = rent[lo] >> 16, cl2 = rent[hi - 1] >> 16;
                    if (tab) {
                        // a table bucket holds more than 16 rows: within the tile it is
                        // a prefix or a suffix
                        if (is_tab(cf)) lo = roff[cf + 1];
                        if (is_tab(cl2)) hi = roff[cl2];
                        if (lo < hi) {
                            cf = rent[lo] >> 16;
                            cl2 = rent[hi - 1] >> 16;
                        }
                    }
                    plan_beg[i] = 0;
                    if (lo < hi) {
                        // start at a multiple of 4 (aligned entry loads); the extra
                        // partners belong to earlier buckets and are masked by their codes
                        const int pb = poff[cf] & ~3, pe = poff[cl2 + 1];
                        plan_beg[i] = pb;
                        cnt[j] = (pe - pb + 15) >> 4;
                    }
                }
                local += cnt[j];
            }
            // inclusive scan of the counts: within each wave by shuffles, then the
            // totals of the waves before it (one barrier)
            int incl = local;
#pragma unroll
            for (int s = 1; s < 64; s <<= 1) {
                const int v = __shfl_up(incl, s);
                if (lane >= s) incl += v;
            }
            if (lane == 63) scan_tmp[wave] = incl;
            __syncthreads();
            for (int w = 0; w < wave; w++) incl += scan_tmp[w];
            int run = incl - local;
#pragma unroll
            for (int j = 0; j < PER; j++) {
                const int i = tid * PER + j;
                if (i < nt) plan_x[i] = run;
                run += cnt[j];
            }
            if (tid == kPassThreads - 1) plan_x[nt] = incl;
            // the run's row entries (16-byte copies; entries past n_r are sentinels)
            for (int i = tid; i < nt * 4; i += kPassThreads) {
                uint4 e4 = ld<uint4>(rent, static_cast<uint32_t>(T0 * 16 + 4 * i) * 4);
                if (tab) {
                    auto mark = [&](uint32_t e) { return is_tab(e >> 16) ? (kSkipCode << 16) | (e & 0xFFFFu) : e; };
                    e4.x = mark(e4.x); e4.y = mark(e4.y); e4.z = mark(e4.z); e4.w = mark(e4.w);
                }
                reinterpret_cast<uint4 *>(row_ent)[i] = e4;
            }
            __syncthreads();
        }
        // ---- this wave's tiles: a contiguous run holding about a quarter of the sub-tiles
        const int total = uni(plan_x[nt]);
        auto lower = [&](int64_t target4) {  // smallest i in [0, nt] with 4 x[i] >= target4
            int lo = 0, hi = nt;
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (4 * static_cast<int64_t>(uni(plan_x[mid])) >= target4) hi = mid; else lo = mid + 1;
            }
            return lo;
        };
        const int tlo = wave == 0 ? 0 : lower(static_cast<int64_t>(wave) * total);
        const int thi = wave == kPassWaves - 1 ? nt : lower(static_cast<int64_t>(wave + 1) * total);
        const int jbeg = uni(plan_x[tlo]), jend = uni(plan_x[thi]);

        auto row_entry = [&](int t) { return row_ent[t * 16 + c]; };
        auto row_entries4 = [&](int t) { return reinterpret_cast<const uint4 *>(row_ent)[t * 4 + q]; };
        auto tile_ents = [&](int t) { return static_cast<const uint32_t *>(row_ent + t * 16); };
        auto row_count = [&](int t) { return min(16, n_r - (T0 + t) * 16); };
        // tiles with no partner at all still own partial rows: they are zero
        auto zero_tiles = [&](int ta, int tb) {
            const floatx4 z[4] = {};
            for (int t = ta; t < tb; t++)
                store_tile<HI1>(tile, part, plow, pexp, ex_lds, ex_in_lds, a.m, HI1, tile_ents(t), row_count(t), q, cl, g,
                           c, z, 0.f);
        };
        // sub-tile j of the run: its tile (searched forward from t) and first partner
        auto tile_of = [&](int j, int t) {
            while (uni(plan_x[t + 1]) <= j) t++;
            return t;
        };
        auto first_partner = [&](int j, int t) { return uni(plan_beg[t]) + 16 * (j - uni(plan_x[t])); };
        auto pent4 = [&](int y) { return ld<uint4>(pent, static_cast<uint32_t>(y + 4 * q) * 4); };

        if (jbeg == jend) {
            zero_tiles(tlo, thi);
        } else {
            // pipeline: partner and row entries two sub-tiles ahead, operands one ahead
            // (sub-tiles past the run load from partner 0 and are never computed).
            // The per-sub-tile state rotates through three slots with the loop unrolled
            // three times, so no register that a load is still filling is ever copied
            // (a copy would make the compiler wait for that load).
            struct Slot {
                int t;        // its tile (wave-uniform)
                uint4 pe;     // entries of its partners 4q .. 4q+3
                uint4 rw[4];  // its tile's rows, loaded when the tile starts here
                uint4 rb[4];  // (*YOSO) the same rows' own b vectors
                int ex;       // e_c with ||a_c|| < 2^e_c for the lane's row c of the tile
            };
            auto fill = [&](Slot &sl, int t, int y, bool new_tile) {
                sl.t = t;
                sl.pe = pent4(y);
                if (new_tile) {
                    sl.ex = rexp[row_entry(t) & 0xFFFFu];  // (sentinel rows read row 0)
                    load_row_tile<HI1>(sl.rw, row_entries4(t), arow, cl);
                    if constexpr (STAR) load_row_tile<HI1>(sl.rb, row_entries4(t), brow, cl);
                }
            };
            Slot A, B, C;
            // the prefetch cursor: tile pt holds sub-tiles [plan_x[pt], pxe); sub-tile j
            // of it starts at partner pbase + 16 j (LDS is read only when it changes tile)
            int pt, pxe, pbase;
            auto cursor_at = [&](int t) {
                pt = t;
                pxe = uni(plan_x[t + 1]);
                pbase = uni(plan_beg[t]) - 16 * uni(plan_x[t]);
            };
            {
                const int t0 = tile_of(jbeg, tlo);
                zero_tiles(tlo, t0);
                fill(A, t0, first_partner(jbeg, t0), true);
                int t1 = t0, y1 = 0;
                if (jbeg + 1 < jend) { t1 = tile_of(jbeg + 1, t0); y1 = first_partner(jbeg + 1, t1); }
                fill(B, t1, y1, t1 != t0);
                cursor_at(t1);
            }
            half8 rh[2], rl[2], rbh[2], rbl[2];
            stage_rows<HI1>(A.rw, tile, q, cl, g, c, rh, rl);
            int erow = A.ex;  // ||a_c|| < 2^erow
            if constexpr (STAR) stage_rows_b<HI1>(A.rb, tile, q, cl, g, c, rbh, rbl);
            // one operand buffer: a sub-tile's registers are reloaded with the next
            // sub-tile as soon as they have been written to the tile
            Sub S;
            load_sub<HI1>(S, A.pe, apar, bpar, cl);
            floatx4 outT[4];
#pragma unroll
            for (int dt = 0; dt < 4; dt++) outT[dt] = floatx4{0.f, 0.f, 0.f, 0.f};

            // step j: `cur` is sub-tile j (in S), `nxt` sub-tile j+1, `nn` receives j+2
            auto step = [&](int j, Slot &cur, Slot &nxt, Slot &nn) -> bool {
                const bool has1 = j + 1 < jend, has2 = j + 2 < jend;
                int t2 = nxt.t, y2 = 0;
                if (has2) {
                    if (j + 2 >= pxe) cursor_at(tile_of(j + 2, pt + 1));
                    t2 = pt;
                    y2 = pbase + 16 * (j + 2);
                }
                publish_sub<HI1>(S, tile, q, cl);
                fill(nn, t2, y2, has2 && t2 != nxt.t);
                const bool newtile = !has1 || nxt.t != cur.t;
                if (has1) load_sub<HI1>(S, nxt.pe, apar, bpar, cl);
                compute_sub<STAR, HI1>(tile, cur.pe, rh, rl, rbh, rbl, xscale, static_cast<int>(row_entry(cur.t) >> 16),
                                  ldexpf(1.0f, -2 - erow), g, c, outT);
                if (newtile) {
                    store_tile<HI1>(tile, part, plow, pexp, ex_lds, ex_in_lds, a.m, HI1, tile_ents(cur.t), row_count(cur.t), q, cl,
                               g, c, outT, ldexpf(oscale, erow));
#pragma unroll
                    for (int dt = 0; dt < 4; dt++) outT[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
                    zero_tiles(cur.t + 1, has1 ? nxt.t : thi);
                    if (has1) {
                        stage_rows<HI1>(nxt.rw, tile, q, cl, g, c, rh, rl);
                        erow = nxt.ex;
                        if constexpr (STAR) stage_rows_b<HI1>(nxt.rb, tile, q, cl, g, c, rbh, rbl);
                    }
                }
                return has1;
            };
            for (int j = jbeg;; j += 3) {
                if (!step(j, A, B, C)) break;
                if (!step(j + 1, B, C, A)) break;
                if (!step(j + 2, C, A, B)) break;
            }
        }
        __syncthreads();  // the plan arrays are rewritten for the next run of tiles
    }
    if (ex_in_lds) {
        // every row's exponent is in LDS (the barrier above orders the writes): one
        // coalesced copy of the row, 16 bytes per lane where aligned, else (and for
        // the tail) byte by byte
        const int n16 = (reinterpret_cast<uintptr_t>(pexp) & 15) == 0 ? n_r >> 4 : 0;
        for (int e = tid; e < n16; e += kPassThreads)
            reinterpret_cast<uint4 *>(pexp)[e] = reinterpret_cast<const uint4 *>(ex_lds)[e];
        for (int e = (n16 << 4) + tid; e < n_r; e += kPassThreads) pexp[e] = ex_lds[e];
    }
}

// ---------------------------------------------------------------- table form
// bucket_kernel: one workgroup per (head, hash, side), launched after pass_kernel,
// for the buckets that take the table form (table_bucket).  Each wave takes whole
// buckets, one after another, from a counter shared by the workgroup:
//   build  M = sum_y a'_y b_y^T (64 x 64) over the bucket's partners, 32 at a time:
//          the group is staged in the wave's LDS tile and all sixteen 16x16 blocks
//          of M accumulate on 16x16x32 MFMAs (three fp16 products each).  The
//          contraction runs over the staged rows, so both operands are read
//          transposed (ds_read_b64_tr_b16).  Entries are fetched two groups ahead
//          and partner rows one group ahead.
//   scale  one power of two brings max |M| below 2^14; M^T is split into fp16
//          (hi, lo), passed through the tile and kept in registers.
//   apply  the bucket's rows, 16 at a time: out^T = M^T A_x^T, stored as the rows'
//          partials like a pass tile; entries two tiles ahead, rows one tile ahead.
// The result for a row is the pass kernel's sum over the same partners, added in
// another order.  No barrier follows the bucket list: the waves share nothing else.
// HI1 (bf16 inputs): a bf16 value scaled by a power of two is an fp16 number
// whenever it lies in fp16's normal range (every value above 2^-27 of its head's
// largest), so its lo part is zero: only the hi parts are read (half the operand
// bytes), M takes one product and the apply two.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kBuildRows = 32;                 // partners per build step
constexpr int kStageBytes = kBuildRows * 512;  // a wave's tile: staged rows [a' hi | a' lo | b hi | b lo]

template <bool HI1>
__global__ __launch_bounds__(kPassThreads, 2) void bucket_kernel(PassArgs a) {
    __shared__ __align__(16) unsigned char stage_lds[kPassWaves * kStageBytes];
    __shared__ __align__(16) uint32_t tent_lds[kPassWaves * 16];  // each wave's tile entries
    __shared__ int16_t list[4096];                                 // the unit's table buckets
    __shared__ int list_n, list_next;

    const int64_t units = a.bh * a.m;
    const int64_t id = xcd_remap(blockIdx.x, 2 * units);
    const int64_t unit = id >> 1;
    const bool kside = id & 1;
    const int64_t b = unit / a.m;
    const int h = static_cast<int>(unit - b * a.m);
    // roles as in pass_kernel: dQ rows = queries (a = dY), partners = keys (a' = V, b = K);
    // dK rows = keys (a = V), partners = queries (a' = dY, b = Q)
    const int n_r = static_cast<int>(kside ? a.k.n : a.q.n);
    const int n_p = static_cast<int>(kside ? a.q.n : a.k.n);
    const int nb = 1 << a.tau;
    const uint32_t *rent = (kside ? a.k.ent : a.q.ent) + unit * ent_stride(n_r);
    const uint32_t *pent = (kside ? a.q.ent : a.k.ent) + unit * ent_stride(n_p);
    const int32_t *qo = a.q.off + unit * (nb + 1), *ko = a.k.off + unit * (nb + 1);
    const int32_t *roff = kside ? ko : qo, *poff = kside ? qo : ko;
    const _Float16 *arow = (kside ? a.vs : a.dys) + b * n_r * (2 * D);
    const _Float16 *apar = (kside ? a.dys : a.vs) + b * n_p * (2 * D);
    const _Float16 *bpar = (kside ? a.qs : a.ks) + b * n_p * (2 * D);
    int16_t *part = (kside ? a.pk : a.pq) + ((b * n_r) * a.m + h) * D;
    uint8_t *plow = (kside ? a.lk : a.lq) + ((b * n_r) * a.m + h) * D;
    int8_t *pexp = (kside ? a.ek : a.eq) + (b * a.m + h) * n_r;
    // the operands carry the head scales 2^(13 - e) of a, a' and b
    const int esum = head_exp(a.pmax, b, kside ? 3 : 1) + head_exp(a.pmax, b, kside ? 1 : 3) +
                     head_exp(a.pmax, b, kside ? 0 : 2);

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = uni(tid >> 6);
    const int g = lane >> 4, c = lane & 15;   // MFMA layout
    const int q = lane >> 4, cl = lane & 15;  // coalesced layout
    unsigned char *st = stage_lds + wave * kStageBytes;
    uint32_t *tent = tent_lds + wave * 16;

    if (tid == 0) {
        list_n = 0;
        list_next = 0;
    }
    __syncthreads();
    for (int cb = tid; cb < nb; cb += kPassThreads)
        if (table_bucket(qo[cb + 1] - qo[cb], ko[cb + 1] - ko[cb], a.tab_t))
            list[atomicAdd(&list_n, 1)] = static_cast<int16_t>(cb);
    __syncthreads();
    const int nl = uni(list_n);

    // Transposed reads of the staged partners for a 16x16x32 operand: lane (g, c)
    // needs partners 8g .. 8g+7 at one dim.  Source lane (g, 4 i4 + a4) addresses
    // partner 8g + i4 (first read) or 8g + 4 + i4 (second), dims 4 a4 .. 4 a4 + 3 of
    // the 16-dim block that starts at 16-byte chunk `chunk` of the staged row;
    // partner p sits in half p >> 4 of the tile, row p & 15.
    const int i4 = c >> 2, a4 = c & 3;
    const unsigned char *sp = st + (g >> 1) * (16 * 512);
    const int ra = 8 * (g & 1) + i4;
    auto trpair = [&](int chunk) {
        const uint32_t o = 8 * (a4 & 1);
        const half4 x = tr_load(sp + swz(ra, chunk + (a4 >> 1), 512) + o);
        const half4 y = tr_load(sp + swz(ra + 4, chunk + (a4 >> 1), 512) + o);
        return __builtin_shufflevector(x, y, 0, 1, 2, 3, 4, 5, 6, 7);
    };

    for (;;) {
        int li = 0;
        if (lane == 0) li = atomicAdd(&list_next, 1);
        li = uni(li);
        if (li >= nl) break;
        const int cb = uni(list[li]);
        const int p0 = uni(poff[cb]), p1 = uni(poff[cb + 1]);
        const int r0 = uni(roff[cb]), r1 = uni(roff[cb + 1]);

        // ---- build.  Slot j of lane (q, cl) holds 16-byte chunk lch of staged row
        // slot_row(j), which is partner y0 + that: all 16 chunks of rows 16 (j >> 2) +
        // 4q + (j & 3), or (HI1) the 8 hi chunks of rows 8j + 2q + (cl >> 3).  Slots past
        // the bucket's end load the bucket's first partner and are staged as zeros (bit j
        // of the masks, computed from the position alone): no load is conditional and no
        // loaded value is used before it is needed, so nothing waits for the loads in flight
        constexpr int NJ = HI1 ? 4 : 8;
        const int lch = HI1 ? (cl & 7) : cl;
        auto slot_row = [&](int j) { return HI1 ? 8 * j + 2 * q + (cl >> 3) : 16 * (j >> 2) + 4 * q + (j & 3); };
        unsigned okn = 0, okr = 0;
        auto group_ents = [&](int y0, uint32_t e[NJ]) {
            okn = 0;
#pragma unroll
            for (int j = 0; j < NJ; j++) {
                const int y = y0 + slot_row(j);
                okn |= y < p1 ? 1u << j : 0u;
                e[j] = pent[y < p1 ? y : p0];
            }
        };
        u32x4 av[NJ], bv[NJ];
        auto group_rows = [&](const uint32_t e[NJ]) {
            okr = okn;
#pragma unroll
            for (int j = 0; j < NJ; j++) {
                const uint32_t off = (e[j] & 0xFFFFu) * (4 * D) + 16 * lch;
                av[j] = ld<u32x4>(apar, off);
                bv[j] = ld<u32x4>(bpar, off);
            }
        };
        floatx4 acc[4][4];
#pragma unroll
        for (int fi = 0; fi < 4; fi++)
#pragma unroll
            for (int ei = 0; ei < 4; ei++) acc[fi][ei] = floatx4{0.f, 0.f, 0.f, 0.f};
        const int ngrp = (p1 - p0 + kBuildRows - 1) / kBuildRows;
        uint32_t en[NJ];
        group_ents(p0, en);
        group_rows(en);
        if (ngrp > 1) group_ents(p0 + kBuildRows, en);
        for (int gi = 0; gi < ngrp; gi++) {
#pragma unroll
            for (int j = 0; j < NJ; j++) {
                const int rr = slot_row(j);
                unsigned char *half_tile = st + (rr >> 4) * (16 * 512);
                const u32x4 keep = u32x4(0u - ((okr >> j) & 1u));  // all ones or all zeros
                lds_st(half_tile, swz(rr & 15, lch, 512), av[j] & keep);
                lds_st(half_tile, swz(rr & 15, 16 + lch, 512), bv[j] & keep);
            }
            if (gi + 1 < ngrp) group_rows(en);
            if (gi + 2 < ngrp) group_ents(p0 + (gi + 2) * kBuildRows, en);
            // A = A'^T (rows f, from the a' part), B = B_y (columns e, from the b part)
            half8 bh[4], bl[4];
#pragma unroll
            for (int ei = 0; ei < 4; ei++) {
                bh[ei] = trpair(16 + 2 * ei);
                if constexpr (!HI1) bl[ei] = trpair(24 + 2 * ei);
            }
#pragma unroll
            for (int fi = 0; fi < 4; fi++) {
                const half8 ah = trpair(2 * fi);
#pragma unroll
                for (int ei = 0; ei < 4; ei++)
                    acc[fi][ei] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bh[ei], acc[fi][ei], 0, 0, 0);
                if constexpr (!HI1) {
                    const half8 al = trpair(8 + 2 * fi);
#pragma unroll
                    for (int ei = 0; ei < 4; ei++)
                        acc[fi][ei] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bl[ei], acc[fi][ei], 0, 0, 0);
#pragma unroll
                    for (int ei = 0; ei < 4; ei++)
                        acc[fi][ei] = __builtin_amdgcn_mfma_f32_16x16x32_f16(al, bh[ei], acc[fi][ei], 0, 0, 0);
                }
            }
        }

        // ---- scale: lane (g, c) of block (fi, ei) holds M[16 fi + 4g + i][16 ei + c]
        float mx = 0.f;
#pragma unroll
        for (int fi = 0; fi < 4; fi++)
#pragma unroll
            for (int ei = 0; ei < 4; ei++)
#pragma unroll
                for (int i = 0; i < 4; i++) mx = fmaxf(mx, fabsf(acc[fi][ei][i]));
        // max |M| < 2^em: M 2^(14 - em) is below 2^14, a normal fp16 pair
        const int em = pow2_above(wave_max(mx));
        const float msc = ldexpf(1.0f, 14 - em);
        // M^T through the tile: row e = 16 ei + c (group ei of 16 rows, 256 bytes each),
        // dims f = 16 fi + 4g + (0..3): 8 bytes of chunk 2 fi + (g >> 1) (hi) and of
        // chunk 8 + that (lo).  (The tile's last transposed reads come first: one
        // wave's LDS accesses execute in order.)
#pragma unroll
        for (int fi = 0; fi < 4; fi++)
#pragma unroll
            for (int ei = 0; ei < 4; ei++) {
                const float v[4] = {acc[fi][ei][0], acc[fi][ei][1], acc[fi][ei][2], acc[fi][ei][3]};
                half4 hi, lo;
                split4_pow2(v, msc, hi, lo);
                unsigned char *grp = st + ei * (16 * 256);
                lds_st(grp, swz(c, 2 * fi + (g >> 1), 256) + 8 * (g & 1), hi);
                lds_st(grp, swz(c, 8 + 2 * fi + (g >> 1), 256) + 8 * (g & 1), lo);
            }
        // M^T as the A operand: lane (g, c) = row e = 16 dt + c, dims 32 kb + 8g + [0, 8)
        half8 mth[4][2], mtl[4][2];
#pragma unroll
        for (int dt = 0; dt < 4; dt++)
#pragma unroll
            for (int kb = 0; kb < 2; kb++) {
                mth[dt][kb] = lds_ld<half8>(st + dt * (16 * 256), swz(c, 4 * kb + g, 256));
                mtl[dt][kb] = lds_ld<half8>(st + dt * (16 * 256), swz(c, 8 + 4 * kb + g, 256));
            }
        // out = s * outT * 2^(e_a + e_a' + e_b - 39) * 2^(em - 14)
        const float orow = ldexpf(a.scale, esum - 39 + em - 14);

        // ---- apply.  Lane (q, cl) loads chunk cl of rows 4q .. 4q+3 of a tile; slots
        // past the bucket's end repeat its first row and are not stored.  A tile's
        // entries are fetched two tiles ahead and its rows one tile ahead, every load
        // unconditional (past the last tile: the last tile again) and the per-tile
        // state rotating through three slots with the loop unrolled three times, so
        // no register that a load is still filling is ever copied
        const int ntile = (r1 - r0 + 15) >> 4;
        // slot i of lane (q, cl): all 16 chunks of row 4q + i, or (HI1) hi chunk cl & 7
        // of row 8i + 2q + (cl >> 3)
        constexpr int NI = HI1 ? 2 : 4;
        auto tile_row = [&](int i) { return HI1 ? 8 * i + 2 * q + (cl >> 3) : 4 * q + i; };
        struct ASlot {
            uint32_t e[NI];
            uint4 r[NI];
        };
        auto tile_ents = [&](int t, uint32_t e[NI]) {
            const int pos = r0 + 16 * min(t, ntile - 1);
#pragma unroll
            for (int i = 0; i < NI; i++) e[i] = rent[pos + tile_row(i) < r1 ? pos + tile_row(i) : pos];
        };
        auto tile_rows = [&](const uint32_t e[NI], uint4 r[NI]) {
#pragma unroll
            for (int i = 0; i < NI; i++) r[i] = ld<uint4>(arow, (e[i] & 0xFFFFu) * (4 * D) + 16 * (HI1 ? (cl & 7) : cl));
        };
        ASlot A, B, C;
        tile_ents(0, A.e);
        tile_rows(A.e, A.r);
        tile_ents(1, B.e);
        auto astep = [&](int t, ASlot &cur, ASlot &nxt, ASlot &nn) -> bool {
            tile_rows(nxt.e, nxt.r);
            tile_ents(t + 2, nn.e);
            const int nvalid = min(16, r1 - (r0 + 16 * t));
            half8 rh[2], rl[2];
            if constexpr (HI1) {
                // the rows' hi chunks into the tile, then the B-operand layout of the hi part
#pragma unroll
                for (int i = 0; i < NI; i++) lds_st(st, swz(tile_row(i), cl & 7, 256), cur.r[i]);
#pragma unroll
                for (int kb = 0; kb < 2; kb++) rh[kb] = lds_ld<half8>(st, swz(c, kb * 4 + g, 256));
                if ((cl & 7) == 0) {
#pragma unroll
                    for (int i = 0; i < NI; i++) tent[tile_row(i)] = cur.e[i];
                }
            } else {
                stage_rows<false>(cur.r, st, q, cl, g, c, rh, rl);
                if (cl == 0) reinterpret_cast<uint4 *>(tent)[q] = make_uint4(cur.e[0], cur.e[1], cur.e[2], cur.e[3]);
            }
            floatx4 outT[4];
#pragma unroll
            for (int dt = 0; dt < 4; dt++) outT[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kb = 0; kb < 2; kb++)
#pragma unroll
                for (int dt = 0; dt < 4; dt++)
                    outT[dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(mth[dt][kb], rh[kb], outT[dt], 0, 0, 0);
            if constexpr (!HI1) {
#pragma unroll
                for (int kb = 0; kb < 2; kb++)
#pragma unroll
                    for (int dt = 0; dt < 4; dt++)
                        outT[dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(mth[dt][kb], rl[kb], outT[dt], 0, 0, 0);
            }
#pragma unroll
            for (int kb = 0; kb < 2; kb++)
#pragma unroll
                for (int dt = 0; dt < 4; dt++)
                    outT[dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(mtl[dt][kb], rh[kb], outT[dt], 0, 0, 0);
            store_tile<HI1>(st, part, plow, pexp, nullptr, false, a.m, a.p16, tent, nvalid, q, cl, g, c, outT, orow);
            return t + 1 < ntile;
        };
        for (int t = 0;; t += 3) {
            if (!astep(t, A, B, C)) break;
            if (!astep(t + 1, B, C, A)) break;
            if (!astep(t + 2, C, A, B)) break;
        }
    }
}

// Q, K, V, dY -> fp16 (hi, lo) rows [hi 64 | lo 64] for the pair passes, each
// head's tensor scaled by 2^(13 - e) (max |x| < 2^e over that tensor of that head),
// so that the largest value lands in [2^12, 2^13) and hi, lo stay normal fp16
// numbers for every value within about 2^-20 of it.  One thread per 8 values.
template <bool BF16>
__global__ __launch_bounds__(256) void split_kernel(const void *__restrict__ q, const void *__restrict__ k,
                                                    const void *__restrict__ v, const void *__restrict__ dy,
                                                    _Float16 *__restrict__ qs, _Float16 *__restrict__ ks,
                                                    _Float16 *__restrict__ vs, _Float16 *__restrict__ dys,
                                                    int8_t *__restrict__ rexq, int8_t *__restrict__ rexk,
                                                    const float *__restrict__ pmax, int64_t bh, int64_t n_q,
                                                    int64_t n_k) {
    const int64_t rows_q = bh * n_q, rows_k = bh * n_k;
    const int64_t per_q = rows_q * (D / 8), per_k = rows_k * (D / 8);
    const int64_t total = 2 * (per_q + per_k);
    for (int64_t tid = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; tid < total;
         tid += static_cast<int64_t>(gridDim.x) * 256) {
        // which: 0 = Q, 1 = dY (query side), 2 = K, 3 = V (key side), the tensor
        // numbering of absmax_kernel
        int which;
        int64_t t;
        if (tid < per_q) { which = 0; t = tid; }
        else if (tid < 2 * per_q) { which = 1; t = tid - per_q; }
        else if (tid < 2 * per_q + per_k) { which = 2; t = tid - 2 * per_q; }
        else { which = 3; t = tid - 2 * per_q - per_k; }
        const void *src = which == 0 ? q : which == 1 ? dy : which == 2 ? k : v;
        _Float16 *dst = which == 0 ? qs : which == 1 ? dys : which == 2 ? ks : vs;
        const int64_t row = t / (D / 8);
        const int64_t head = row / (which < 2 ? n_q : n_k);
        const float scale = ldexpf(1.0f, 13 - head_exp(pmax, head, which));
        const int o = static_cast<int>(t - row * (D / 8)) * 8;
        float x[8];
        load8<BF16>(src, row * D + o, x);
        half8 hi, lo;
        split8(x, scale, hi, lo);
        *reinterpret_cast<half8 *>(dst + row * (2 * D) + o) = hi;
        // bf16 inputs: the lo halves are zero (wherever the scaled value is a normal
        // fp16 number) and the pair passes read hi halves only
        if constexpr (!BF16) *reinterpret_cast<half8 *>(dst + row * (2 * D) + D + o) = lo;
        // rows of dY and V (the rows a of the pair passes): e with ||a|| < 2^e, from the
        // fp16 pairs the products use.  A row is 8 consecutive threads (every tensor
        // and the grid stride are multiples of 8 threads, so the 8 are all active).
        float ss = 0.f;
#pragma unroll
        for (int i = 0; i < 8; i++) {
            const float xv = static_cast<float>(hi[i]) + (BF16 ? 0.f : static_cast<float>(lo[i]));
            ss = fmaf(xv, xv, ss);
        }
        ss += __shfl_xor(ss, 1, 8);
        ss += __shfl_xor(ss, 2, 8);
        ss += __shfl_xor(ss, 4, 8);
        if ((which & 1) && o == 0) {
            // ss < 2^e2  ->  ||a|| < 2^ceil(e2 / 2); the sum's rounding (far below one
            // part in 2^20) is covered by the factor 4 of slack in the 2^14 bound of S
            int e2 = 0;
            if (ss > 0.f) frexpf(ss, &e2);
            (which == 1 ? rexq : rexk)[row] = static_cast<int8_t>((e2 + 1) >> 1);
        }
    }
}

// out[r][:] = sum_h M[r][h][:] * 2^(e[r][h] - 22), M = (high part) * 256 + (low byte)
// - 2^22, in hash order; 8 lanes per row, 8 values each.  The hashes go in groups of
// eight, each group's loads issued before the previous group is added, so that a
// lane keeps up to 384 bytes in flight.
template <bool BF16>
__global__ __launch_bounds__(kReduceThreads) void reduce_kernel(const int16_t *__restrict__ part,
                                                                const uint8_t *__restrict__ plow,
                                                                const int8_t *__restrict__ pexp,
                                                                void *__restrict__ out, int64_t rows, int64_t n,
                                                                int m) {
    const int64_t r = (static_cast<int64_t>(blockIdx.x) * kReduceThreads + threadIdx.x) >> 3;
    const int q = threadIdx.x & 7;
    if (r >= rows) return;
    typedef unsigned int uint4v __attribute__((ext_vector_type(4)));
    typedef unsigned int uint2v __attribute__((ext_vector_type(2)));
    const uint4v *src = reinterpret_cast<const uint4v *>(part + r * m * D) + q;
    const uint2v *srl = reinterpret_cast<const uint2v *>(plow + r * m * D) + q;
    const int64_t b = r / n;
    const int8_t *ex = pexp + b * m * n + (r - b * n);
    float s[8];
#pragma unroll
    for (int i = 0; i < 8; i++) s[i] = 0.f;
    // 24-bit rows: M = high * 256 + low - 2^22, value = M 2^(e - 22), e from the exponent
    // array.  bf16 outputs take 16-bit rows (no low parts): value = high 2^(e - 15),
    // except values 0 .. 3, whose two low bits hold bits 2j, 2j+1 of e and whose
    // value is (high >> 2) 2^(e - 13); the thread of a row holding values 0 .. 7
    // decodes e and the row's other seven threads take it from there
    auto add = [&](const uint4v &v, const uint2v &l, int e) {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
        if constexpr (BF16) {
            const uint32_t eb = (w[0] & 3u) | ((w[0] >> 14) & 0xCu) | ((w[1] & 3u) << 4) | ((w[1] >> 10) & 0xC0u);
            e = __shfl(static_cast<int>(static_cast<int8_t>(eb)), 0, 8);
        }
        const float sc = ldexpf(1.0f, e - (BF16 ? 15 : 22));
        const uint32_t lb[2] = {l.x, l.y};
#pragma unroll
        for (int i = 0; i < 8; i++) {
            const uint32_t hu = (w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
            int mv;
            if constexpr (BF16) {
                mv = static_cast<int16_t>(hu);
                if (i < 4 && q == 0) mv = (mv >> 2) * 4;  // the exponent bits out, the 14-bit value scaled to 16
            } else {
                mv = static_cast<int>((hu << 8) | ((lb[i >> 2] >> (8 * (i & 3))) & 0xFFu)) - (1 << 22);
            }
            s[i] = fmaf(static_cast<float>(mv), sc, s[i]);  // |M| <= 2^22: exact in fp32
        }
    };
    // groups of eight hashes, double-buffered: group g+1 is loaded while g is added
    uint4v v[2][8];
    uint2v l[2][8];
    int e[2][8];
    auto load = [&](uint4v w[8], uint2v lw[8], int f[8], int h0) {
#pragma unroll
        for (int u = 0; u < 8; u++) w[u] = __builtin_nontemporal_load(src + (h0 + u) * (D / 8));
        if constexpr (!BF16) {
#pragma unroll
            for (int u = 0; u < 8; u++) lw[u] = __builtin_nontemporal_load(srl + (h0 + u) * (D / 8));
        }
#pragma unroll
        for (int u = 0; u < 8; u++) f[u] = BF16 ? 0 : ex[(h0 + u) * n];
    };
    const int ng = m >> 3;
    if (ng > 0) load(v[0], l[0], e[0], 0);
    for (int g = 0; g < ng; g += 2) {
        if (g + 1 < ng) load(v[1], l[1], e[1], 8 * (g + 1));
#pragma unroll
        for (int u = 0; u < 8; u++) add(v[0][u], l[0][u], e[0][u]);
        if (g + 1 < ng) {
            if (g + 2 < ng) load(v[0], l[0], e[0], 8 * (g + 2));
#pragma unroll
            for (int u = 0; u < 8; u++) add(v[1][u], l[1][u], e[1][u]);
        }
    }
    int h = 8 * ng;
    for (; h < m; h++)
        add(__builtin_nontemporal_load(src + h * (D / 8)), BF16 ? uint2v{0u, 0u} : __builtin_nontemporal_load(srl + h * (D / 8)),
            BF16 ? 0 : ex[h * n]);
    if constexpr (BF16) {
        uint4 o;
        o.x = static_cast<uint32_t>(f32_to_bf16(s[0])) | (static_cast<uint32_t>(f32_to_bf16(s[1])) << 16);
        o.y = static_cast<uint32_t>(f32_to_bf16(s[2])) | (static_cast<uint32_t>(f32_to_bf16(s[3])) << 16);
        o.z = static_cast<uint32_t>(f32_to_bf16(s[4])) | (static_cast<uint32_t>(f32_to_bf16(s[5])) << 16);
        o.w = static_cast<uint32_t>(f32_to_bf16(s[6])) | (static_cast<uint32_t>(f32_to_bf16(s[7])) << 16);
        reinterpret_cast<uint4 *>(static_cast<uint16_t *>(out) + r * D)[q] = o;
    } else {
        float4 *o = reinterpret_cast<float4 *>(static_cast<float *>(out) + r * D) + 2 * q;
        o[0] = make_float4(s[0], s[1], s[2], s[3]);
        o[1] = make_float4(s[4], s[5], s[6], s[7]);
    }
}

__global__ void zero_kernel(uint32_t *__restrict__ p, int64_t count) {
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < count;
         e += static_cast<int64_t>(gridDim.x) * blockDim.x)
        p[e] = 0u;
}

// ---------------------------------------------------------------- dense form (short sequences)
// eq. (pseudo-gradient-q) with the hashes summed first: C = sum_h B_h (C_ij is the
// number of hashes under which q_i and k_j collide), then
//   dQ = tau/(2m) [(dY V^T) .* C] K,     dK = tau/(2m) [(dY V^T) .* C]^T Q,
// every (query, key) pair of a head visited once in dense 16 x 16 MFMA blocks.
// With a few rows per bucket (short sequences) the pair tiles above are nearly
// empty; this form does n_q n_k (2d + d) multiply-adds per side with full tiles,
// needs no fp16 copies, no partial rows and no reduction.
//
// One workgroup (4 waves) per (head, 64 fixed rows, side), both sides in one
// launch.  dQ: fixed = queries (a = dY), streamed = keys (g = V, y = K); dK: fixed =
// keys (a = V), streamed = queries (g = dY, y = Q), and there also dV = (1/m) C^T dY
// from the same staged dY rows (eq. gradient-v with the hashes summed first).
//   1. C[fixed row][streamed row] as bytes in LDS from the streamed side's bucket
//      lists (sort_kernel): for each fixed row and hash, +1 at every streamed row
//      of the fixed row's bucket (counts <= m <= 64 fit a byte).
//   2. the fixed rows' a in the MFMA B layout, each row scaled by 2^(13 - e_a).
//   3. streamed tiles of 64 rows: g and y rows staged in LDS, each tile scaled by
//      2^(13 - e) from its largest |value|; per 16 x 16 block G^T = g a^T (three
//      fp16 products), W = G .* C tau/(2m) 2^-(16 + k), out^T += y^T W.  The
//      accumulators are rescaled exactly when a tile's scales change.
constexpr int kDenseRows = 64;     // fixed rows per workgroup (16 per wave)
// Fewer fixed-row blocks than this and a longest side of at least kDenseSplitMinRows:
// each block's streamed rows are shared among up to kDenseSplit workgroups.
constexpr int64_t kDenseSplitBelow = 128;
constexpr int64_t kDenseSplitMinRows = 256;
constexpr int kDenseSplit = 8;
constexpr int kDenseTile = 64;     // streamed rows per LDS tile
constexpr int kDenseMaxN = 1024;   // streamed rows whose counts fit in LDS

// u32 words per fixed row of the count matrix: a multiple of 64 plus 4, so that
// the 16 rows x 4 words a block reads (rows c, words 4g / 4 + ...) hit distinct banks
__host__ __device__ constexpr int dense_stride(int64_t n_s) {
    return static_cast<int>(((n_s + 3) / 4 + 63) / 64 * 64 + 4);
}

struct DenseSide {
    const uint16_t *fcodes;  // fixed side's codes [bh][n_f][m]
    const uint32_t *sent;    // streamed side's sorted entries [bh*m][ent_stride(n_s)]
    const int32_t *soff;     // streamed side's bucket offsets [bh*m][2^tau + 1]
    const void *fa;          // fixed side's a rows [bh][n_f][64]
    const void *sg, *sy;     // streamed side's g rows and y rows [bh][n_s][64]
    void *out;               // [bh][n_f][64]: dQ or dK
    void *out2;              // [bh][n_f][64]: dV (key side), else nullptr
    float *pout, *pout2;     // split > 1: fp32 partial outputs [split][bh][n_f][64] of out, out2
    int64_t n_f, n_s;
};

struct DenseArgs {
    DenseSide side[2];       // 0: dQ (queries fixed), 1: dK and dV (keys fixed)
    int64_t bh;
    int m, tau;
    int split;               // workgroups per fixed-row block, each streaming a contiguous share of the rows
};

template <bool BF16>
__device__ __forceinline__ void dense_store(void *dst, int64_t off, const floatx4 &o, float sc) {
    if constexpr (BF16) {
        uint2 w2;
        w2.x = static_cast<uint32_t>(f32_to_bf16(o[0] * sc)) | (static_cast<uint32_t>(f32_to_bf16(o[1] * sc)) << 16);
        w2.y = static_cast<uint32_t>(f32_to_bf16(o[2] * sc)) | (static_cast<uint32_t>(f32_to_bf16(o[3] * sc)) << 16);
        *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(dst) + off) = w2;
    } else {
        *reinterpret_cast<float4 *>(static_cast<float *>(dst) + off) =
            make_float4(o[0] * sc, o[1] * sc, o[2] * sc, o[3] * sc);
    }
}

template <bool BF16, int TILE>
__global__ __launch_bounds__(256, TILE == 32 ? 3 : 2) void dense_kernel(DenseArgs args) {
    // staging: RPW rows per wave, LPR lanes per row, DPL dims per lane
    constexpr int RPW = TILE / 4, LPR = 64 / RPW, DPL = D / LPR;
    extern __shared__ __align__(16) uint32_t cnt[];  // [kDenseRows][dense_stride(n_s)]
    __shared__ __align__(16) unsigned char g_lds[TILE * 256];
    __shared__ __align__(16) unsigned char y_lds[TILE * 256];
    __shared__ float tmax[8];

    // blocks of side 0, then side 1 (both sides' tile counts)
    const int64_t t0 = (args.side[0].n_f + kDenseRows - 1) / kDenseRows;
    const int64_t t1 = (args.side[1].n_f + kDenseRows - 1) / kDenseRows;
    const int split = args.split;
    const int64_t blk0 = xcd_remap(blockIdx.x, args.bh * (t0 + t1) * split);
    const int sp = static_cast<int>(blk0 % split);
    const int64_t blk = blk0 / split;
    const bool kside = blk >= args.bh * t0;
    const DenseSide a = args.side[kside ? 1 : 0];
    const int64_t tiles_f = kside ? t1 : t0;
    const int64_t lblk = kside ? blk - args.bh * t0 : blk;
    const int64_t b = lblk / tiles_f;
    const int r0 = static_cast<int>(lblk - b * tiles_f) * kDenseRows;
    const int m = args.m, tau = args.tau;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c = lane & 15;
    const int stride = dense_stride(a.n_s);
    const int nf = static_cast<int>(a.n_f), ns = static_cast<int>(a.n_s);
    // the streamed rows of this workgroup: [cs0, cs1), whole tiles (split > 1: a share of
    // them, the fp32 partial outputs summed afterwards by dense_sum_kernel)
    const int slen = ((ns + split - 1) / split + TILE - 1) / TILE * TILE;
    const int cs0 = min(ns, sp * slen), cs1 = min(ns, cs0 + slen);

    // the streamed side's rows: lane l of wave w loads row RPW w + (l % RPW), dims
    // DPL (l / RPW) + [0, DPL) of a tile (rows clamped: the prefetch past the last
    // tile reads the last rows again and is never used).  The first tile's loads are
    // in flight while the counts are built.
    const int lrow = RPW * wave + (lane % RPW), lq = lane / RPW;
    auto load_tile = [&](int c0, float (&xg)[DPL], float (&xy)[DPL]) {
        const int64_t off = (b * a.n_s + min(c0 + lrow, ns - 1)) * D + DPL * lq;
#pragma unroll
        for (int u = 0; u < DPL / 8; u++) {
            load8<BF16>(a.sg, off + 8 * u, xg + 8 * u);
            load8<BF16>(a.sy, off + 8 * u, xy + 8 * u);
        }
    };
    float xga[DPL], xya[DPL], xgb[DPL], xyb[DPL];
    load_tile(cs0, xga, xya);

    // ---- 1. collision counts.  Items (fixed row, hash) in groups of eight per
    // thread: their codes, then their bucket ranges, then the entries, each stage's
    // loads all in flight before the next stage uses them.
    for (int e = tid; e < kDenseRows * stride; e += 256) cnt[e] = 0u;
    __syncthreads();
    {
        const int B = 1 << tau;
        const int64_t es = ent_stride(a.n_s);
        const int items = kDenseRows * m;
        constexpr int U = 8;
        for (int i0 = tid; i0 < items; i0 += 256 * U) {
            int beg[U], len[U], r[U];
            int64_t unit[U];
            int code[U];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int item = min(i0 + 256 * u, items - 1);
                r[u] = item / m;
                const int h = item - r[u] * m;
                unit[u] = b * m + h;
                code[u] = a.fcodes[(b * a.n_f + min(r0 + r[u], nf - 1)) * m + h] & (B - 1);
            }
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int32_t *off = a.soff + unit[u] * (B + 1) + code[u];
                beg[u] = off[0];
                len[u] = off[1];
            }
            int most = 0;
#pragma unroll
            for (int u = 0; u < U; u++) {
                const bool ok = i0 + 256 * u < items && r0 + r[u] < nf;
                len[u] = ok ? len[u] - beg[u] : 0;
                most = max(most, len[u]);
            }
            for (int p = 0; p < most; p++) {
                uint32_t j[U];
#pragma unroll
                for (int u = 0; u < U; u++) j[u] = a.sent[unit[u] * es + beg[u] + min(p, max(len[u] - 1, 0))];
#pragma unroll
                for (int u = 0; u < U; u++) {
                    if (p < len[u]) {
                        const uint32_t jj = j[u] & 0xFFFFu;
                        atomicAdd(&cnt[r[u] * stride + (jj >> 2)], 1u << (8 * (jj & 3)));
                    }
                }
            }
        }
    }

    // ---- 2. the fixed rows' a: lane (g, c) holds row r0 + 16 wave + c, dims kb*32 + 8g + [0, 8)
    const int frow = r0 + wave * 16 + c;
    half8 arh[2], arl[2];
    int ea = 0;
    {
        float y[2][8];
        const int64_t off = (b * a.n_f + min(frow, nf - 1)) * D;
        load8<BF16>(a.fa, off + 8 * g, y[0]);
        load8<BF16>(a.fa, off + 32 + 8 * g, y[1]);
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

    // ---- 3. streamed tiles of TILE rows (32 rows, two 16 x 16 blocks, where there are
    // enough workgroups to fill the GPU: smaller tiles and fewer prefetch registers
    // leave room for three workgroups per CU; else 64).  Staging as the loads.
    auto put_row = [&](unsigned char *dst, const float x[DPL], float scale) {
#pragma unroll
        for (int u = 0; u < DPL / 8; u++) {
            half8 h, l;
            split8(x + 8 * u, scale, h, l);
            *reinterpret_cast<half8 *>(dst + swz(lrow, (DPL / 8) * lq + u, 256)) = h;
            *reinterpret_cast<half8 *>(dst + swz(lrow, 8 + (DPL / 8) * lq + u, 256)) = l;
        }
    };
    // rows past the range become zeros when the tile is staged
    auto row_max = [&](int c0, float x[DPL]) {
        const bool ok = c0 + lrow < cs1;
        float mx = 0.f;
#pragma unroll
        for (int i = 0; i < DPL; i++) {
            x[i] = ok ? x[i] : 0.f;
            mx = fmaxf(mx, fabsf(x[i]));
        }
        return mx;
    };
    const int pr = 4 * g + (c >> 2), a4 = c & 3;
    const floatx4 z4 = {0.f, 0.f, 0.f, 0.f};
    floatx4 out[4], out2[4];
#pragma unroll
    for (int dt = 0; dt < 4; dt++) out[dt] = out2[dt] = z4;
    // tau/(2m) G C is scaled by 2^-(16 + k), 2^k >= tau: |G| < 2^32 after the row and
    // tile scalings and C <= m, so the weight stays below 2^15; dV's weight C/m is
    // scaled by 2^15 (at most 2^15)
    int k2 = 0;
    while ((1 << k2) < tau) k2++;
    const float wgd = static_cast<float>(tau) / (2.0f * static_cast<float>(m)) * ldexpf(1.0f, -(16 + k2));
    const float wvd = 32768.0f / static_cast<float>(m);
    const bool with_dv = a.out2 != nullptr;
    // for m a power of two the weight C 2^15 / m (C <= m) is an exact fp16 number: its
    // lo half is zero and so is the product with it
    const bool wv_exact = (m & (m - 1)) == 0;
    const uint32_t *crow = cnt + (16 * wave + c) * stride;  // the lane's fixed row of counts
    int eg = 0, ey = 0;
    // one streamed tile from (xg, xy), the next one's loads into (gn, yn) (two
    // register sets, swapped by unrolling the loop twice: copying registers a load
    // is still filling would wait for it)
    auto do_tile = [&](int c0, float (&xg)[DPL], float (&xy)[DPL], float (&gn)[DPL], float (&yn)[DPL]) {
        __syncthreads();  // counts complete (first tile); the previous tile has been read
        float mg = row_max(c0, xg);
        float my = row_max(c0, xy);
        mg = wave_max(mg);
        my = wave_max(my);
        if (lane == 0) {
            tmax[wave] = mg;
            tmax[4 + wave] = my;
        }
        __syncthreads();
        const int eg_new = pow2_above(fmaxf(fmaxf(tmax[0], tmax[1]), fmaxf(tmax[2], tmax[3])));
        const int ey_new = pow2_above(fmaxf(fmaxf(tmax[4], tmax[5]), fmaxf(tmax[6], tmax[7])));
        put_row(g_lds, xg, ldexpf(1.0f, 13 - eg_new));
        put_row(y_lds, xy, ldexpf(1.0f, 13 - ey_new));
        // (rescaled only when a tile scale changed: a factor of 1 would change nothing)
        if (c0 > cs0 && (eg != eg_new || ey != ey_new)) {
            const float f = ldexpf(1.0f, eg + ey - eg_new - ey_new), f2 = ldexpf(1.0f, eg - eg_new);
#pragma unroll
            for (int dt = 0; dt < 4; dt++) {
                out[dt] *= f;
                out2[dt] *= f2;
            }
        }
        eg = eg_new;
        ey = ey_new;
        load_tile(c0 + TILE, gn, yn);
        __syncthreads();
#pragma unroll 1
        for (int cb = 0; cb < TILE / 16; cb++) {
            if (c0 + 16 * cb >= cs1) break;
            // G^T block: lane (g, c) = (g row c0 + 16cb + 4g + i) . (a row c)
            half8 bh[2], bl[2];
#pragma unroll
            for (int kb = 0; kb < 2; kb++) {
                bh[kb] = lds_ld<half8>(g_lds, swz(16 * cb + c, kb * 4 + g, 256));
                bl[kb] = lds_ld<half8>(g_lds, swz(16 * cb + c, 8 + kb * 4 + g, 256));
            }
            floatx4 s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(bh[0], arh[0], z4, 0, 0, 0);
            floatx4 s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(bh[1], arh[1], z4, 0, 0, 0);
            s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(bh[0], arl[0], s0, 0, 0, 0);
            s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(bh[1], arl[1], s1, 0, 0, 0);
            s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(bl[0], arh[0], s0, 0, 0, 0);
            s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(bl[1], arh[1], s1, 0, 0, 0);
            const floatx4 gt = s0 + s1;
            // counts of streamed rows c0 + 16cb + 4g .. +3 against the lane's fixed row
            const uint32_t cw = crow[(c0 + 16 * cb + 4 * g) >> 2];
            float w[4];
#pragma unroll
            for (int i = 0; i < 4; i++) w[i] = gt[i] * static_cast<float>((cw >> (8 * i)) & 0xFFu) * wgd;
            half4 wh, wl;
            split4(w, 1.0f, wh, wl);
            // y^T of the block as the A operand (lane (g, c): dim 16dt + c, rows 4g .. 4g+3)
            half4 yh[4], yl[4];
#pragma unroll
            for (int dt = 0; dt < 4; dt++) {
                yh[dt] = tr_load(y_lds + swz(16 * cb + pr, 2 * dt + (a4 >> 1), 256) + 8 * (a4 & 1));
                yl[dt] = tr_load(y_lds + swz(16 * cb + pr, 8 + 2 * dt + (a4 >> 1), 256) + 8 * (a4 & 1));
            }
            // hi*lo + lo*hi as one 16x16x32 product over [y hi | y lo] and [w lo ; w hi],
            // then hi*hi
            const half8 wlh = __builtin_shufflevector(wl, wh, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
            for (int dt = 0; dt < 4; dt++) {
                const half8 yt = __builtin_shufflevector(yh[dt], yl[dt], 0, 1, 2, 3, 4, 5, 6, 7);
                out[dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(yt, wlh, out[dt], 0, 0, 0);
            }
#pragma unroll
            for (int dt = 0; dt < 4; dt++) out[dt] = __builtin_amdgcn_mfma_f32_16x16x16f16(yh[dt], wh, out[dt], 0, 0, 0);
            if (with_dv) {
                // dV^T += dY^T (C / m) 2^15: the staged g rows are dY on this side
                float wv[4];
#pragma unroll
                for (int i = 0; i < 4; i++) wv[i] = static_cast<float>((cw >> (8 * i)) & 0xFFu) * wvd;
                half4 vh, vl;
                if (wv_exact) {
#pragma unroll
                    for (int i = 0; i < 4; i++) vh[i] = static_cast<_Float16>(wv[i]);
                } else {
                    split4(wv, 1.0f, vh, vl);
                }
                half4 gh[4], gl[4];
#pragma unroll
                for (int dt = 0; dt < 4; dt++) {
                    gh[dt] = tr_load(g_lds + swz(16 * cb + pr, 2 * dt + (a4 >> 1), 256) + 8 * (a4 & 1));
                    gl[dt] = tr_load(g_lds + swz(16 * cb + pr, 8 + 2 * dt + (a4 >> 1), 256) + 8 * (a4 & 1));
                }
#pragma unroll
                for (int dt = 0; dt < 4; dt++)
                    out2[dt] = __builtin_amdgcn_mfma_f32_16x16x16f16(gh[dt], vh, out2[dt], 0, 0, 0);
                if (!wv_exact) {
#pragma unroll
                    for (int dt = 0; dt < 4; dt++)
                        out2[dt] = __builtin_amdgcn_mfma_f32_16x16x16f16(gh[dt], vl, out2[dt], 0, 0, 0);
                }
#pragma unroll
                for (int dt = 0; dt < 4; dt++)
                    out2[dt] = __builtin_amdgcn_mfma_f32_16x16x16f16(gl[dt], vh, out2[dt], 0, 0, 0);
            }
        }
    };
    for (int c0 = cs0; c0 < cs1; c0 += 2 * TILE) {
        do_tile(c0, xga, xya, xgb, xyb);
        if (c0 + TILE < cs1) do_tile(c0 + TILE, xgb, xyb, xga, xya);
    }

    // ---- 4. out = acc 2^(16 + k) (a row 2^(13 - e_a)) (g tile 2^(13 - e_g)) (y tile 2^(13 - e_y));
    // dV = acc2 2^-15 (g tile 2^(13 - e_g)); lane (g, c) holds out[fixed row c][16dt + 4g + i]
    if (frow < nf) {
        const float sc = ldexpf(1.0f, 16 + k2 + ea - 13 + eg - 13 + ey - 13);
        const float sc2 = ldexpf(1.0f / 32768.0f, eg - 13);
#pragma unroll
        for (int dt = 0; dt < 4; dt++) {
            const int64_t off = (b * a.n_f + frow) * D + 16 * dt + 4 * g;
            if (split == 1) {
                dense_store<BF16>(a.out, off, out[dt], sc);
                if (with_dv) dense_store<BF16>(a.out2, off, out2[dt], sc2);
            } else {
                const int64_t po = sp * (args.bh * a.n_f * D) + off;
                *reinterpret_cast<floatx4 *>(a.pout + po) = out[dt] * sc;
                if (with_dv) *reinterpret_cast<floatx4 *>(a.pout2 + po) = out2[dt] * sc2;
            }
        }
    }
}

// dQ, dK, dV = sums over the splits of their fp32 partial outputs, in split order
// (four values per thread, the three outputs one after another), stored as fp32 or bf16.
struct DenseSum {
    const float *part[3];
    void *out[3];
    int64_t count4[3];  // four-value groups per output (a split's partials are count4 groups apart)
    int split;
};

template <bool BF16>
__global__ __launch_bounds__(256) void dense_sum_kernel(DenseSum a) {
    const int64_t total = a.count4[0] + a.count4[1] + a.count4[2];
    for (int64_t t = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; t < total;
         t += static_cast<int64_t>(gridDim.x) * 256) {
        const int o = t < a.count4[0] ? 0 : (t < a.count4[0] + a.count4[1] ? 1 : 2);
        const int64_t i = t - (o > 0 ? a.count4[0] : 0) - (o > 1 ? a.count4[1] : 0);
        const float *part = o == 0 ? a.part[0] : (o == 1 ? a.part[1] : a.part[2]);
        floatx4 acc = reinterpret_cast<const floatx4 *>(part)[i];
        for (int sp = 1; sp < a.split; sp++) acc += reinterpret_cast<const floatx4 *>(part)[sp * a.count4[o] + i];
        dense_store<BF16>(o == 0 ? a.out[0] : (o == 1 ? a.out[1] : a.out[2]), 4 * i, acc, 1.0f);
    }
}

// ---------------------------------------------------------------- dense forward (short sequences)
// Y = (1/m) sum_h B_h V (Sec. 3.1, 3.2) with the hashes summed first: Y = (1/m) C V,
// C_ij the number of hashes under which q_i and k_j collide, every (query, key)
// pair of a head visited once.  C is counted from the two rows' codes and C V runs
// on 16 x 16 MFMA blocks (C is an exact fp16 integer, V an fp16 (hi, lo) pair).  At
// a few rows per bucket the bucket tables cost a fixed amount per table and feature
// slice that this form does not have; it does n_q n_k (~1.5 tau + 1 compares + 2d
// multiply-adds) of work per head.
//
// Codes as bit planes: plane t of a row is the bit vector over its hashes of bit t
// of each code (one 32-bit word per 32 hashes), so that for a (query, key) pair the
// hashes on which the codes differ are OR_t (plane_t(q) ^ plane_t(k)) and
// C = m - popcount of that.  A tile's codes are copied into LDS as they lie in
// memory (one coalesced run) and each thread assembles whole plane words of a row.
//
// One workgroup (4 waves) per (head, 64 queries): wave w owns queries 16w .. 16w+15,
// lane (g, c) query 16w + c.  Keys stream through LDS in tiles of 64 (V rows split
// into fp16 (hi, lo) under the tile's power-of-two scale; planes); per 16-key block
// lane (g, c) counts C for its query against keys 4g .. 4g+3 and out^T += V^T C.
constexpr int kDenseFwdMaxN = 1024;   // both sides at most this many rows: dense forward

// Plane row stride in words: tau * PW words rounded up to a 16-byte multiple, plus
// 16 bytes (the words between are zero)
__host__ __device__ constexpr int plane_stride(int tau, int pw) { return (tau * pw + 3) / 4 * 4 + 4; }

// Raw codes of rows [r0, r0 + 64) of a [rows][m] array (64 m contiguous uint16, one
// coalesced run): thread t loads elements t + 256 i, clamped to the array.
template <int PW>
struct RawCodes {
    uint32_t c[8 * PW];
};

template <int PW>
__device__ __forceinline__ void load_raw_codes(RawCodes<PW> &rc, const uint16_t *codes, int r0, int nrows, int m,
                                               int tid) {
    const int last = nrows * m - 1, base = r0 * m;
#pragma unroll
    for (int i = 0; i < 8 * PW; i++) rc.c[i] = codes[min(base + tid + 256 * i, last)];
}

// LDS copy of the raw codes: row r at uint16 offset r * raw_stride (16-byte
// aligned rows whose 16-byte reads by 16 consecutive rows hit distinct banks).
template <int PW>
__host__ __device__ constexpr int raw_stride() { return 64 * PW + 8; }

template <int PW>
__device__ __forceinline__ void store_raw_codes(const RawCodes<PW> &rc, uint16_t *dst, int m, float inv_m, int tid) {
#pragma unroll
    for (int i = 0; i < 8 * PW; i++) {
        const int e = tid + 256 * i;
        if (e < 64 * m) {
            // e / m, exact: (e + 1/2) / m lies at least 1/(2m) from an integer and the
            // product's rounding error is below 2^-16 for e < 2^12
            const int r = static_cast<int>((static_cast<float>(e) + 0.5f) * inv_m);
            dst[r * raw_stride<PW>() + (e - r * m)] = static_cast<uint16_t>(rc.c[i]);
        }
    }
}

// Planes of the 64 rows in LDS (row stride `ps` words: word t*PW + w of a row holds
// bits [32w, 32w + 32) of plane t).  Thread t builds planes (t >> 6) + 4k of row
// t & 63 from the row's codes, two operations per code and plane.
template <int PW>
__device__ __forceinline__ void build_planes(const uint16_t *raw, int m, int tau, int ps, uint32_t *dst, int tid) {
    const int r = tid & 63, p0 = tid >> 6;
    const uint4 *src = reinterpret_cast<const uint4 *>(raw + r * raw_stride<PW>());
#pragma unroll
    for (int w = 0; w < PW; w++) {
        uint32_t cw[16];  // codes 32w .. 32w + 31, two per word
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const uint4 q4 = src[4 * w + j];
            cw[4 * j] = q4.x;
            cw[4 * j + 1] = q4.y;
            cw[4 * j + 2] = q4.z;
            cw[4 * j + 3] = q4.w;
        }
        // hashes past m (the rest of the row's LDS slot) are masked out
        const int valid = m - 32 * w;
        const uint32_t keep = valid >= 32 ? 0xFFFFFFFFu : valid <= 0 ? 0u : (1u << valid) - 1u;
#pragma unroll
        for (int k = 0; k < 3; k++) {
            const int t = p0 + 4 * k;
            if (t < tau) {
                uint32_t word = 0u;
#pragma unroll
                for (int j = 0; j < 16; j++) {
                    word |= __builtin_amdgcn_ubfe(cw[j], t, 1) << (2 * j);
                    word |= __builtin_amdgcn_ubfe(cw[j], 16 + t, 1) << (2 * j + 1);
                }
                dst[r * ps + t * PW + w] = word & keep;
            }
        }
    }
}

template <bool BF16, int PW>
__global__ __launch_bounds__(256) void dense_fwd_kernel(const uint16_t *__restrict__ qcodes,
                                                        const uint16_t *__restrict__ kcodes,
                                                        const void *__restrict__ v, void *__restrict__ y, int64_t bh,
                                                        int n_q, int n_k, int m, int tau) {
    constexpr int NW = 12 * PW;  // plane words per row at most (tau <= 12)
    __shared__ __align__(16) unsigned char v_lds[kDenseTile * 256];
    __shared__ __align__(16) uint32_t kp_lds[kDenseTile * plane_stride(12, PW)];
    __shared__ __align__(16) uint32_t qp_lds[kDenseRows * plane_stride(12, PW)];
    __shared__ __align__(16) uint16_t raw_lds[64 * raw_stride<PW>()];
    __shared__ float tmax[4];

    const int64_t tiles = (n_q + kDenseRows - 1) / kDenseRows;
    const int64_t blk = xcd_remap(blockIdx.x, bh * tiles);
    const int64_t b = blk / tiles;
    const int r0 = static_cast<int>(blk - b * tiles) * kDenseRows;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c = lane & 15;
    const int ps = plane_stride(tau, PW);
    const int nw = tau * PW;  // plane words per row
    const float inv_m = 1.0f / static_cast<float>(m);
    const uint16_t *kc = kcodes + b * n_k * m;

    // plane words past tau * PW are read as zeros and never written
    for (int i = tid; i < kDenseTile * plane_stride(12, PW); i += 256) kp_lds[i] = qp_lds[i] = 0u;

    // staging of V: lane l of wave w stages row 16w + (l & 15), dims 16 (l >> 4) + [0, 16)
    const int lrow = 16 * wave + (lane & 15), lq = lane >> 4;
    // a key tile's V rows and raw codes, loaded together (rows clamped: the prefetch
    // past the last tile reads the last rows again and is never used)
    auto load_tile = [&](int c0, RawCodes<PW> &rc, float (&x)[16]) {
        const int64_t off = (b * n_k + min(c0 + lrow, n_k - 1)) * D + 16 * lq;
        load8<BF16>(v, off, x);
        load8<BF16>(v, off + 8, x + 8);
        load_raw_codes<PW>(rc, kc, c0, n_k, m, tid);
    };
    RawCodes<PW> kca, kcb;
    float xa[16], xb[16];
    if (n_k > 0) load_tile(0, kca, xa);

    // ---- the workgroup's queries as planes; lane (g, c) keeps query 16 wave + c's
    uint32_t qp[NW];
    {
        RawCodes<PW> rc;
        load_raw_codes<PW>(rc, qcodes + b * n_q * m, r0, n_q, m, tid);
        store_raw_codes<PW>(rc, raw_lds, m, inv_m, tid);
        __syncthreads();
        build_planes<PW>(raw_lds, m, tau, ps, qp_lds, tid);
        __syncthreads();
        const uint4 *src = reinterpret_cast<const uint4 *>(qp_lds + (16 * wave + c) * ps);
#pragma unroll
        for (int j = 0; j < NW / 4; j++) {
            const uint4 w4 = j * 4 < nw ? src[j] : make_uint4(0u, 0u, 0u, 0u);
            qp[4 * j] = w4.x;
            qp[4 * j + 1] = w4.y;
            qp[4 * j + 2] = w4.z;
            qp[4 * j + 3] = w4.w;
        }
    }

    const int pr = 4 * g + (c >> 2), a4 = c & 3;
    const floatx4 z4 = {0.f, 0.f, 0.f, 0.f};
    floatx4 out[4];
#pragma unroll
    for (int dt = 0; dt < 4; dt++) out[dt] = z4;
    int ev = 0;
    // one key tile from (rc, x), the next one's loads into (rn, xn) (two register
    // sets, swapped by unrolling the loop twice: copying registers a load is still
    // filling would wait for it)
    auto do_tile = [&](int c0, RawCodes<PW> &rc, float (&x)[16], RawCodes<PW> &rn, float (&xn)[16]) {
        __syncthreads();  // the previous tile (and the query planes' raw codes) have been read
        store_raw_codes<PW>(rc, raw_lds, m, inv_m, tid);
        float mx = 0.f;
        {
            const bool ok = c0 + lrow < n_k;
#pragma unroll
            for (int i = 0; i < 16; i++) {
                x[i] = ok ? x[i] : 0.f;
                mx = fmaxf(mx, fabsf(x[i]));
            }
        }
        mx = wave_max(mx);
        if (lane == 0) tmax[wave] = mx;
        __syncthreads();
        // planes of the tile's keys (keys past n_k have zero V rows, so their codes,
        // clamped copies of the last key's, do not matter)
        build_planes<PW>(raw_lds, m, tau, ps, kp_lds, tid);
        const int ev_new = pow2_above(fmaxf(fmaxf(tmax[0], tmax[1]), fmaxf(tmax[2], tmax[3])));
        {
            half8 h[2], l[2];
            const float sc = ldexpf(1.0f, 13 - ev_new);
            split8(x, sc, h[0], l[0]);
            split8(x + 8, sc, h[1], l[1]);
#pragma unroll
            for (int u = 0; u < 2; u++) {
                *reinterpret_cast<half8 *>(v_lds + swz(lrow, 2 * lq + u, 256)) = h[u];
                *reinterpret_cast<half8 *>(v_lds + swz(lrow, 8 + 2 * lq + u, 256)) = l[u];
            }
        }
        if (c0 > 0) {
            const float f = ldexpf(1.0f, ev - ev_new);
#pragma unroll
            for (int dt = 0; dt < 4; dt++) out[dt] *= f;
        }
        ev = ev_new;
        load_tile(c0 + kDenseTile, rn, xn);
        __syncthreads();
#pragma unroll 1
        for (int cb = 0; cb < kDenseTile / 16; cb++) {
            if (c0 + 16 * cb >= n_k) break;
            // C for the lane's query against keys 16cb + 4g + i
            half4 ch;
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const uint4 *src = reinterpret_cast<const uint4 *>(kp_lds + (16 * cb + 4 * g + i) * ps);
                uint32_t d0 = 0u, d1 = 0u;
#pragma unroll
                for (int j = 0; j < NW / 4; j++) {
                    if (j * 4 < nw) {
                        const uint4 w4 = src[j];
                        const uint32_t kw[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
                        for (int u = 0; u < 4; u++) {
                            // word 4j + u: plane (4j + u) / PW, hash word (4j + u) % PW
                            const uint32_t dx = qp[4 * j + u] ^ kw[u];
                            if (PW == 1 || (u & 1) == 0)
                                d0 |= dx;
                            else
                                d1 |= dx;
                        }
                    }
                }
                const int cnt = m - static_cast<int>(__builtin_popcount(d0) + __builtin_popcount(d1));
                ch[i] = static_cast<_Float16>(static_cast<float>(cnt));
            }
            // V^T of the block as the A operand (lane (g, c): dim 16dt + c, keys 4g .. 4g+3)
            half4 vh[4], vl[4];
#pragma unroll
            for (int dt = 0; dt < 4; dt++) {
                vh[dt] = tr_load(v_lds + swz(16 * cb + pr, 2 * dt + (a4 >> 1), 256) + 8 * (a4 & 1));
                vl[dt] = tr_load(v_lds + swz(16 * cb + pr, 8 + 2 * dt + (a4 >> 1), 256) + 8 * (a4 & 1));
            }
#pragma unroll
            for (int dt = 0; dt < 4; dt++) out[dt] = __builtin_amdgcn_mfma_f32_16x16x16f16(vh[dt], ch, out[dt], 0, 0, 0);
#pragma unroll
            for (int dt = 0; dt < 4; dt++) out[dt] = __builtin_amdgcn_mfma_f32_16x16x16f16(vl[dt], ch, out[dt], 0, 0, 0);
        }
    };
    for (int c0 = 0; c0 < n_k; c0 += 2 * kDenseTile) {
        do_tile(c0, kca, xa, kcb, xb);
        if (c0 + kDenseTile < n_k) do_tile(c0 + kDenseTile, kcb, xb, kca, xa);
    }

    // Y = out 2^(e_v - 13) / m; lane (g, c) holds out[query c][16dt + 4g + i]
    const int frow = r0 + 16 * wave + c;
    if (frow < n_q) {
        const float sc = ldexpf(1.0f, ev - 13) / static_cast<float>(m);
#pragma unroll
        for (int dt = 0; dt < 4; dt++) dense_store<BF16>(y, (b * n_q + frow) * D + 16 * dt + 4 * g, out[dt], sc);
    }
}

unsigned elementwise_grid(int64_t count) {
    const int64_t blocks = (count + 255) / 256;
    return static_cast<unsigned>(blocks < 8192 ? (blocks > 0 ? blocks : 1) : 8192);
}

size_t align_up(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

template <bool BF16>
hipError_t launch_reduce(const int16_t *part, const uint8_t *plow, const int8_t *pexp, void *out, int64_t rows,
                         int64_t n, int m, hipStream_t stream) {
    if (rows == 0) return hipSuccess;
    const int64_t blocks = (rows * 8 + kReduceThreads - 1) / kReduceThreads;
    KernelTimer timer("reduce_kernel", stream);
    hipLaunchKernelGGL(reduce_kernel<BF16>, dim3(static_cast<unsigned>(blocks)), dim3(kReduceThreads), 0, stream,
                       part, plow, pexp, out, rows, n, m);
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

// hi1: the inputs are bf16, so the fp16 lo parts of their scaled copies are zero (see
// load_sub) and both forms read hi parts only.
hipError_t launch_pass(const PassArgs &a, int64_t units, bool star, bool hi1, hipStream_t stream) {
    const dim3 grid(static_cast<unsigned>(2 * units)), block(kPassThreads);
    if (star) {
        KernelTimer timer("pass_star_kernel", stream);
        if (hi1)
            hipLaunchKernelGGL((pass_kernel<true, true>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((pass_kernel<true, false>), grid, block, 0, stream, a);
    } else {
        {
            KernelTimer timer("pass_kernel", stream);
            if (hi1)
                hipLaunchKernelGGL((pass_kernel<false, true>), grid, block, 0, stream, a);
            else
                hipLaunchKernelGGL((pass_kernel<false, false>), grid, block, 0, stream, a);
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess || a.tab_t == 0) return e;
        // after the pass: the pass blocks write their whole exponent rows, the table
        // buckets' entries included, and these writes must land last
        KernelTimer timer("bucket_kernel", stream);
        if (hi1)
            hipLaunchKernelGGL(bucket_kernel<true>, dim3(static_cast<unsigned>(2 * units)), dim3(kPassThreads), 0,
                               stream, a);
        else
            hipLaunchKernelGGL(bucket_kernel<false>, dim3(static_cast<unsigned>(2 * units)), dim3(kPassThreads), 0,
                               stream, a);
    }
    return hipGetLastError();
}

// *YOSO's derived codes: for every (row, hash h, bit t < tau) the code of hash h
// with bit t removed, a (tau-1)-bit code: out[r][h*tau + t] = (c >> (t+1)) << t |
// (c & (2^t - 1)).  Two rows collide under it exactly when their codes agree on
// every bit but t, so the pair passes over these m*tau hashes count, per pair and
// hash, the bits whose removal makes the codes agree.
__global__ void drop_bit_kernel(const uint16_t *__restrict__ codes, uint16_t *__restrict__ out, int64_t rows, int m,
                                int tau) {
    const int64_t total = rows * m * tau;
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < total;
         e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t r = e / (m * tau);
        const int ht = static_cast<int>(e - r * m * tau);
        const int h = ht / tau, t = ht - h * tau;
        const uint32_t c = codes[r * m + h] & ((1u << tau) - 1u);
        out[e] = static_cast<uint16_t>(((c >> (t + 1)) << t) | (c & ((1u << t) - 1u)));
    }
}

}  // namespace

BackwardLayout backward_layout(bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m, int tau) {
    BackwardLayout L;
    const int64_t units = bh * m;
    const size_t nb = (static_cast<size_t>(1) << tau) + 1;
    size_t o = 0;
    L.qoff = o; o = align_up(o + units * nb * 4);
    L.koff = o; o = align_up(o + units * nb * 4);
    L.qent = o; o = align_up(o + units * ent_stride(n_q) * 4);
    L.kent = o; o = align_up(o + units * ent_stride(n_k) * 4);
    L.qct = o; o = align_up(o + static_cast<size_t>(units) * n_q * 2);
    L.kct = o; o = align_up(o + static_cast<size_t>(units) * n_k * 2);
    L.qs = o; o = align_up(o + static_cast<size_t>(bh) * n_q * D * 4);
    L.dys = o; o = align_up(o + static_cast<size_t>(bh) * n_q * D * 4);
    L.ks = o; o = align_up(o + static_cast<size_t>(bh) * n_k * D * 4);
    L.vs = o; o = align_up(o + static_cast<size_t>(bh) * n_k * D * 4);
    L.pq = o; o = align_up(o + static_cast<size_t>(bh) * n_q * m * D * 2);
    L.pk = o; o = align_up(o + static_cast<size_t>(bh) * n_k * m * D * 2);
    // the low parts of the 24-bit partial rows (bf16 outputs take 16-bit rows: none)
    const size_t low = bf16 ? 0 : static_cast<size_t>(D);
    L.lq = o; o = align_up(o + static_cast<size_t>(bh) * n_q * m * low);
    L.lk = o; o = align_up(o + static_cast<size_t>(bh) * n_k * m * low);
    // exponents of 24-bit rows (16-bit rows carry theirs)
    const size_t ex = bf16 ? 0 : 1;
    L.eq = o; o = align_up(o + ex * bh * n_q * m);
    L.ek = o; o = align_up(o + ex * bh * n_k * m);
    L.rexq = o; o = align_up(o + static_cast<size_t>(bh) * n_q);
    L.rexk = o; o = align_up(o + static_cast<size_t>(bh) * n_k);
    L.pmax = o; o = align_up(o + static_cast<size_t>(bh) * 4 * kMaxParts * 4);
    L.table = o; o = align_up(o + table_workspace_bytes(bf16, bh, n_k, m, tau));
    L.total = o;
    return L;
}

namespace {

// The dense form serves short sequences (both sides at most kDenseMaxN rows);
// *YOSO always takes the pair passes.
bool dense_form(int64_t n_q, int64_t n_k, bool star) { return !star && n_q <= kDenseMaxN && n_k <= kDenseMaxN; }

// dQ and dK from codes with m hashes of tau bits: bucket sort, per-head maxima,
// the fp16 split, the pair passes (weights of *YOSO when `star`) and the hash sums;
// for short sequences the dense form instead, which also writes dV.  `L` is
// backward_layout(bf16, bh, n_q, n_k, m, tau) within `ws`.
hipError_t launch_pairs(const uint16_t *qcodes, const uint16_t *kcodes, const void *q, const void *k, const void *v,
                        const void *dy, bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m, int tau, float scale,
                        bool star, void *dq, void *dk, void *dv, const BackwardLayout &L, unsigned char *ws,
                        hipStream_t stream) {
    hipError_t e;
    const int64_t units = bh * m;
    if (units == 0) return hipSuccess;
    const int64_t ebytes = bf16 ? 2 : 4;
    if (n_q == 0 || n_k == 0) {
        // no pairs: dq and dk are zero
        if ((e = zero_output(dq, bh * n_q * D * ebytes, stream)) != hipSuccess) return e;
        return zero_output(dk, bh * n_k * D * ebytes, stream);
    }

    {
        // Sort modes, by what fits in a workgroup's LDS: (1) the column's codes (read
        // once, with stride m) and its sorted entries staged, 6 bytes per row; (2) the
        // codes transposed to [bh][m][n] first (each block then reads its column
        // contiguously) and the entries staged, 4 bytes per row; (3) transposed codes,
        // entries stored straight to memory (eight waves when tau <= 10).  Short
        // sequences take mode (1) with one wave per block.
        const int64_t n_max = n_q > n_k ? n_q : n_k;
        const bool narrow = n_max <= kSortNarrowN && 2 * units >= kSortNarrowBlocks;
        size_t sort_lds = sort_base_lds(narrow ? kSortThreadsNarrow : kSortThreads, tau);
        const bool stage_codes = sort_lds + static_cast<size_t>(n_max) * 6 <= kSortStageLds;
        const bool stage_ent = stage_codes || sort_lds + static_cast<size_t>(n_max) * 4 <= kSortEntLds;
        const bool transposed = !stage_codes;
        sort_lds += stage_codes ? static_cast<size_t>(n_max) * 6 : stage_ent ? static_cast<size_t>(n_max) * 4 : 0;
        const bool wide = !stage_ent && tau <= 10;
        uint16_t *qct = reinterpret_cast<uint16_t *>(ws + L.qct), *kct = reinterpret_cast<uint16_t *>(ws + L.kct);
        if (transposed) {
            for (int side = 0; side < 2; side++) {
                const int64_t n = side ? n_k : n_q;
                const int64_t items = bh * ((n + 63) / 64) * ((m + 63) / 64);
                const unsigned blocks = static_cast<unsigned>(items < 65536 ? items : 65536);
                KernelTimer timer("codes_t_kernel", stream);
                const uint16_t *src = side ? kcodes : qcodes;
                if (m % 8 == 0 && (reinterpret_cast<uintptr_t>(src) & 15) == 0)
                    hipLaunchKernelGGL(codes_t_kernel<true>, dim3(blocks), dim3(256), 0, stream,
                                       side ? kcodes : qcodes, side ? kct : qct, bh, n, m);
                else
                    hipLaunchKernelGGL(codes_t_kernel<false>, dim3(blocks), dim3(256), 0, stream,
                                       side ? kcodes : qcodes, side ? kct : qct, bh, n, m);
                if ((e = hipGetLastError()) != hipSuccess) return e;
            }
        }
        const uint16_t *qsrc = transposed ? qct : qcodes, *ksrc = transposed ? kct : kcodes;
        KernelTimer timer("sort_kernel", stream);
        const dim3 grid(static_cast<unsigned>(2 * units));
        int32_t *qo = reinterpret_cast<int32_t *>(ws + L.qoff), *ko = reinterpret_cast<int32_t *>(ws + L.koff);
        uint32_t *qe = reinterpret_cast<uint32_t *>(ws + L.qent), *ke = reinterpret_cast<uint32_t *>(ws + L.kent);
        if (narrow)
            hipLaunchKernelGGL(sort_kernel<kSortThreadsNarrow>, grid, dim3(kSortThreadsNarrow), sort_lds, stream, qsrc,
                               ksrc, m, n_q, n_k, tau, transposed, stage_codes, stage_ent, qo, ko, qe, ke);
        else if (wide)
            hipLaunchKernelGGL(sort_kernel<kSortThreadsWide>, grid, dim3(kSortThreadsWide),
                               sort_base_lds(kSortThreadsWide, tau), stream, qsrc, ksrc, m, n_q, n_k, tau, transposed,
                               false, false, qo, ko, qe, ke);
        else
            hipLaunchKernelGGL(sort_kernel<kSortThreads>, grid, dim3(kSortThreads), sort_lds, stream, qsrc, ksrc, m,
                               n_q, n_k, tau, transposed, stage_codes, stage_ent, qo, ko, qe, ke);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;

    if (dense_form(n_q, n_k, star)) {
        // short sequences: dQ, dK (and dV) from dense blocks masked by the collision counts
        DenseArgs d;
        for (int side = 0; side < 2; side++) {
            DenseSide &ds = d.side[side];
            ds.fcodes = side ? kcodes : qcodes;
            ds.sent = reinterpret_cast<const uint32_t *>(ws + (side ? L.qent : L.kent));
            ds.soff = reinterpret_cast<const int32_t *>(ws + (side ? L.qoff : L.koff));
            ds.fa = side ? v : dy;
            ds.sg = side ? dy : v;
            ds.sy = side ? q : k;
            ds.out = side ? dk : dq;
            ds.out2 = side ? dv : nullptr;
            ds.n_f = side ? n_k : n_q;
            ds.n_s = side ? n_q : n_k;
        }
        d.bh = bh; d.m = m; d.tau = tau;
        const int64_t blocks1 = bh * ((n_q + kDenseRows - 1) / kDenseRows + (n_k + kDenseRows - 1) / kDenseRows);
        // Few fixed-row blocks (a head or two): each block's streamed rows are split
        // among kDenseSplit workgroups, whose fp32 partial outputs go to the workspace
        // after the partial-row sections' start (unused by this form) and are summed in
        // split order.  Many blocks: one workgroup each, outputs stored directly.
        int split = 1;
        const size_t part_room = L.total - L.pq;
        const size_t per_split = static_cast<size_t>(bh) * static_cast<size_t>(n_q + 2 * n_k) * D * sizeof(float);
        if (blocks1 < kDenseSplitBelow && (n_q > n_k ? n_q : n_k) >= kDenseSplitMinRows)
            while (split < kDenseSplit && per_split * (2 * split) <= part_room) split *= 2;
        d.split = split;
        float *pq0 = reinterpret_cast<float *>(ws + L.pq);
        d.side[0].pout = pq0;
        d.side[0].pout2 = nullptr;
        d.side[1].pout = pq0 + static_cast<int64_t>(split) * bh * n_q * D;
        d.side[1].pout2 = d.side[1].pout + static_cast<int64_t>(split) * bh * n_k * D;
        const int64_t blocks = blocks1 * split;
        const size_t lds = static_cast<size_t>(kDenseRows) * dense_stride(n_q > n_k ? n_q : n_k) * 4;
        {
            KernelTimer timer("dense_kernel", stream);
            // 32-row streamed tiles where the blocks fill the GPU at three per CU (384 x
            // 512: 618 -> 515 us), 64-row ones for a few blocks (fewer barriers per row)
            const bool t32 = blocks >= 512;
            auto kernel = bf16 ? (t32 ? dense_kernel<true, 32> : dense_kernel<true, 64>)
                               : (t32 ? dense_kernel<false, 32> : dense_kernel<false, 64>);
            hipLaunchKernelGGL(kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), lds, stream, d);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        if (split == 1) return hipSuccess;
        KernelTimer timer("dense_sum_kernel", stream);
        DenseSum sa;
        sa.part[0] = d.side[0].pout; sa.part[1] = d.side[1].pout; sa.part[2] = d.side[1].pout2;
        sa.out[0] = dq; sa.out[1] = dk; sa.out[2] = dv;
        sa.count4[0] = bh * n_q * D / 4; sa.count4[1] = sa.count4[2] = bh * n_k * D / 4;
        sa.split = split;
        const int64_t total = sa.count4[0] + 2 * sa.count4[1];
        const int64_t grid = (total + 255) / 256 < 4096 ? (total + 255) / 256 : 4096;
        if (bf16)
            hipLaunchKernelGGL(dense_sum_kernel<true>, dim3(static_cast<unsigned>(grid)), dim3(256), 0, stream, sa);
        else
            hipLaunchKernelGGL(dense_sum_kernel<false>, dim3(static_cast<unsigned>(grid)), dim3(256), 0, stream, sa);
        return hipGetLastError();
    }

    _Float16 *qs = reinterpret_cast<_Float16 *>(ws + L.qs), *ks = reinterpret_cast<_Float16 *>(ws + L.ks);
    _Float16 *vs = reinterpret_cast<_Float16 *>(ws + L.vs), *dys = reinterpret_cast<_Float16 *>(ws + L.dys);
    float *pmax = reinterpret_cast<float *>(ws + L.pmax);
    int8_t *rexq = reinterpret_cast<int8_t *>(ws + L.rexq), *rexk = reinterpret_cast<int8_t *>(ws + L.rexk);
    {
        KernelTimer timer("absmax_kernel", stream);
        const dim3 grid(static_cast<unsigned>(bh * 4 * kMaxParts));
        if (bf16)
            hipLaunchKernelGGL(absmax_kernel<true>, grid, dim3(256), 0, stream, q, dy, k, v, n_q, n_k, pmax);
        else
            hipLaunchKernelGGL(absmax_kernel<false>, grid, dim3(256), 0, stream, q, dy, k, v, n_q, n_k, pmax);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    {
        const int64_t threads = 2 * bh * (n_q + n_k) * (D / 8);
        const int64_t blocks = (threads + 255) / 256 < 65536 ? (threads + 255) / 256 : 65536;
        KernelTimer timer("split_kernel", stream);
        if (bf16)
            hipLaunchKernelGGL(split_kernel<true>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, q, k, v,
                               dy, qs, ks, vs, dys, rexq, rexk, pmax, bh, n_q, n_k);
        else
            hipLaunchKernelGGL(split_kernel<false>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, q, k,
                               v, dy, qs, ks, vs, dys, rexq, rexk, pmax, bh, n_q, n_k);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;

    PassArgs a;
    a.q = Side{reinterpret_cast<const uint32_t *>(ws + L.qent), reinterpret_cast<const int32_t *>(ws + L.qoff), n_q};
    a.k = Side{reinterpret_cast<const uint32_t *>(ws + L.kent), reinterpret_cast<const int32_t *>(ws + L.koff), n_k};
    a.qs = qs; a.ks = ks; a.vs = vs; a.dys = dys;
    a.pmax = pmax;
    a.rexq = rexq; a.rexk = rexk;
    a.pq = reinterpret_cast<int16_t *>(ws + L.pq);
    a.pk = reinterpret_cast<int16_t *>(ws + L.pk);
    a.lq = reinterpret_cast<uint8_t *>(ws + L.lq);
    a.lk = reinterpret_cast<uint8_t *>(ws + L.lk);
    a.eq = reinterpret_cast<int8_t *>(ws + L.eq);
    a.ek = reinterpret_cast<int8_t *>(ws + L.ek);
    a.bh = bh; a.m = m; a.tau = tau;
    a.scale = scale;
    a.tab_t = star ? 0 : kTableT;
    a.p16 = bf16;
    e = launch_pass(a, units, star, bf16, stream);
    if (e != hipSuccess) return e;
    if (bf16) {
        if ((e = launch_reduce<true>(a.pq, a.lq, a.eq, dq, bh * n_q, n_q, m, stream)) != hipSuccess) return e;
        return launch_reduce<true>(a.pk, a.lk, a.ek, dk, bh * n_k, n_k, m, stream);
    }
    if ((e = launch_reduce<false>(a.pq, a.lq, a.eq, dq, bh * n_q, n_q, m, stream)) != hipSuccess) return e;
    return launch_reduce<false>(a.pk, a.lk, a.ek, dk, bh * n_k, n_k, m, stream);
}

}  // namespace

int backward_table_threshold() { return kTableT; }

// The dense forward's work grows as n_q n_k, the tables' as (n_q + n_k) plus a cost
// per table of 2^tau m rows; measured on 16-row to 1024-row sequences, the dense
// form is faster where it fills the chip (a workgroup per head and 64 queries: at
// least two per CU) and n_q n_k stays below 2^19 per 8192 table rows per head.
bool dense_forward_applies(int64_t bh, int64_t n_q, int64_t n_k, int m, int tau) {
    if (n_q > kDenseFwdMaxN || n_k > kDenseFwdMaxN) return false;
    if (bh * ((n_q + kDenseRows - 1) / kDenseRows) < 512) return false;
    const int64_t per = (int64_t{1} << tau) * m / 8192;
    return n_q * n_k <= (int64_t{1} << 19) * (per > 1 ? per : 1);
}

hipError_t launch_dense_forward(const uint16_t *qcodes, const uint16_t *kcodes, const void *v, void *y, bool bf16,
                                int64_t bh, int64_t n_q, int64_t n_k, int m, int tau, hipStream_t stream) {
    const int64_t blocks = bh * ((n_q + kDenseRows - 1) / kDenseRows);
    if (blocks == 0) return hipSuccess;
    KernelTimer timer("dense_fwd_kernel", stream);
    const int nq = static_cast<int>(n_q), nk = static_cast<int>(n_k);
    auto kernel = bf16 ? (m > 32 ? dense_fwd_kernel<true, 2> : dense_fwd_kernel<true, 1>)
                       : (m > 32 ? dense_fwd_kernel<false, 2> : dense_fwd_kernel<false, 1>);
    hipLaunchKernelGGL(kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, qcodes, kcodes, v, y, bh,
                       nq, nk, m, tau);
    return hipGetLastError();
}

hipError_t launch_backward(const uint16_t *qcodes, const uint16_t *kcodes, const void *q, const void *k,
                           const void *v, const void *dy, bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m,
                           int tau, void *dq, void *dk, void *dv, void *workspace, hipStream_t stream) {
    const BackwardLayout L = backward_layout(bf16, bh, n_q, n_k, m, tau);
    unsigned char *ws = static_cast<unsigned char *>(workspace);
    // dV: the forward's table machinery with the roles of queries and keys swapped
    // (the dense form of short sequences computes it with dQ, dK)
    const bool dense = dense_form(n_q, n_k, false) && bh > 0 && n_q > 0 && n_k > 0;
    if (!dense) {
        const hipError_t e = launch_table(qcodes, dy, kcodes, dv, bf16, bh, n_q, n_k, m, tau, ws + L.table, stream);
        if (e != hipSuccess) return e;
    }
    return launch_pairs(qcodes, kcodes, q, k, v, dy, bf16, bh, n_q, n_k, m, tau,
                        static_cast<float>(tau) / (2.0f * static_cast<float>(m)), false, dq, dk, dv, L, ws, stream);
}

StarLayout backward_star_layout(bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m, int tau) {
    StarLayout S;
    S.pairs = backward_layout(bf16, bh, n_q, n_k, m * tau, tau - 1);
    size_t o = align_up(S.pairs.total);
    S.qcodes = o; o = align_up(o + static_cast<size_t>(bh) * n_q * m * tau * 2);
    S.kcodes = o; o = align_up(o + static_cast<size_t>(bh) * n_k * m * tau * 2);
    S.table = o; o = align_up(o + table_workspace_bytes(bf16, bh, n_k, m, tau));
    S.total = o;
    return S;
}

hipError_t launch_backward_star(const uint16_t *qcodes, const uint16_t *kcodes, const void *q, const void *k,
                                const void *v, const void *dy, bool bf16, int64_t bh, int64_t n_q, int64_t n_k, int m,
                                int tau, void *dq, void *dk, void *dv, void *workspace, hipStream_t stream) {
    const StarLayout S = backward_star_layout(bf16, bh, n_q, n_k, m, tau);
    unsigned char *ws = static_cast<unsigned char *>(workspace);
    // dV: eq. (gradient-v), as in launch_backward
    hipError_t e = launch_table(qcodes, dy, kcodes, dv, bf16, bh, n_q, n_k, m, tau, ws + S.table, stream);
    if (e != hipSuccess) return e;
    uint16_t *qd = reinterpret_cast<uint16_t *>(ws + S.qcodes), *kd = reinterpret_cast<uint16_t *>(ws + S.kcodes);
    for (int side = 0; side < 2; side++) {
        const int64_t rows = bh * (side ? n_k : n_q);
        if (rows == 0) continue;
        const int64_t total = rows * m * tau;
        KernelTimer timer("drop_bit_kernel", stream);
        hipLaunchKernelGGL(drop_bit_kernel, dim3(elementwise_grid(total)), dim3(256), 0, stream, side ? kcodes : qcodes,
                           side ? kd : qd, rows, m, tau);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    // the pairs of the m*tau derived (tau-1)-bit hashes, each weighted by
    // 1/(pi sqrt(max(1 - x^2, 1/64))) and averaged over the m original hashes
    return launch_pairs(qd, kd, q, k, v, dy, bf16, bh, n_q, n_k, m * tau, tau - 1, 1.0f / static_cast<float>(m), true,
                        dq, dk, nullptr, S.pairs, ws, stream);
}

}  // namespace yoso
