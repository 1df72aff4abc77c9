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
// carries two values at once.  Each value v of feature dim d is quantised to
// q = rint(v 2^k_d) with one power-of-two scale per dim of the workgroup's
// slice, chosen so that 2^k_d times a bound on every bucket sum of |v| of that dim
// stays below 2^30: the dim's sum of |v| over the source rows, or (fp32 outputs of
// more than 8192 source rows, where that sum grows with n_src and the rounding step
// with it) the smaller of that sum and the count of the largest bucket times the
// dim's largest |v|, the counts taken in LDS before the scatter.  A bucket sum of
// rounded values is then below 2^30 + n_src/2 in magnitude.  A dim of small values
// is thus resolved as finely as a dim of large ones.  Two adjacent dims
// (q_lo, q_hi) are packed as the 64-bit integer q_hi 2^32 + q_lo; sums of packed
// words never corrupt each other's field because |sum q_lo| < 2^31.  Integer
// sums are exact and independent of the order of the atomics, so the tables (and
// the outputs) are deterministic.  The only rounding is the quantisation,
// |error| <= 2^-k / 2 per value.
//
// LDS layout: word (c*G + h)*P + p holds dims (2p, 2p+1) of bucket c of hash
// h (P = DS/2 words per row).
//   scatter: one key per instruction; lane (h, p) adds its word of the key into
//            row (code_h, h).  The 32 lanes of a half-wave cover distinct
//            (h, p) in a row block whose stride is a multiple of the 64 LDS
//            banks, so they never conflict.
//   gather:  4 lanes per query (8 for 64 hashes), each reading the whole P-word
//            rows of G/4 hashes in a rotated order (the 16 lanes of a 16-byte
//            access pass hit distinct bank groups), then a DPP butterfly sums
//            the lanes of the query.
#include <type_traits>

#include "common.h"
#include "launch.h"
#include "timing.h"

namespace yoso {

namespace {

constexpr int kTableThreads = 512;
constexpr int kTableWaves = kTableThreads / 64;
// fp32 outputs with more source rows than this also bound the bucket sums by the
// largest bucket count (a count pass over the codes before the scatter)
constexpr int64_t kTableHistRows = 8192;
// launches with fewer workgroups than this take narrower slices (down to two dims)
constexpr int64_t kTableFewBlocks = 128;

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
    int hist;                   // 1: bound the bucket sums by the largest bucket count too
};

// (lo, hi) of a packed word whose fields are signed and |field sums| < 2^31:
// the low dword is lo itself; the high dword is hi minus the borrow of a negative lo.
__device__ __forceinline__ void unpack(unsigned long long w, int &lo, int &hi) {
    lo = static_cast<int>(static_cast<uint32_t>(w));
    hi = static_cast<int>(static_cast<uint32_t>(w >> 32)) + static_cast<int>(static_cast<uint32_t>(lo) >> 31);
}

// KM: how a step broadcasts key values to the lanes: 0 -> one key per step
// (readlane), 1 -> two keys per step (two readlanes), 2 -> more (ds_bpermute).
template <bool BF16, int DS, int KM>
__global__ __launch_bounds__(kTableThreads) void table_kernel(TableArgs a) {
    constexpr int P = DS / 2;   // packed words per table row
    constexpr int S = D / DS;   // slices per head
    extern __shared__ __align__(16) unsigned long long tab[];  // [2^tau][G][P]
    __shared__ float wave_red[kTableWaves * DS];
    __shared__ float wave_mx[kTableWaves * DS];
    __shared__ float dim_sum[DS], dim_max[DS];  // per dim: sum and largest |v| over the source rows
    __shared__ uint32_t wave_cnt[kTableWaves];
    __shared__ int scale_exp[DS];

    const int64_t blocks = a.bh * S;
    const int64_t logical = xcd_remap(blockIdx.x, blocks);
    const int64_t b = logical / S;
    const int slice = static_cast<int>(logical - b * S);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar loops)
    const int G = a.G;
    const int cmask = (1 << a.tau) - 1;
    const int64_t vbase = b * a.n_src * D + slice * DS;

    // ---- scale: for each dim of this slice, the sum of |v| over all source rows
    // bounds every bucket sum of that dim -> exponent k.  With `hist` the count of
    // the largest bucket times the dim's largest |v| bounds them too, and the smaller
    // bound sets k (per pass of hashes, below).
    // (eight rows per thread in flight at once: the pass is latency-bound; rows past
    // the end re-read the last row and add nothing)
    {
        float sa[DS], sm[DS];
#pragma unroll
        for (int d = 0; d < DS; d++) sa[d] = sm[d] = 0.f;
        constexpr int U = 8;
        const int64_t last = a.n_src - 1;
        for (int64_t j0 = tid; j0 < a.n_src; j0 += U * kTableThreads) {
            float v[U][DS];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int64_t j = j0 + u * kTableThreads;
                load_slice<BF16, DS>(a.values, vbase + (j < last ? j : last) * D, v[u]);
            }
#pragma unroll
            for (int u = 0; u < U; u++) {
                const bool in = j0 + u * kTableThreads < a.n_src;
#pragma unroll
                for (int d = 0; d < DS; d++) {
                    sa[d] += in ? fabsf(v[u][d]) : 0.f;
                    sm[d] = fmaxf(sm[d], in ? fabsf(v[u][d]) : 0.f);
                }
            }
        }
#pragma unroll
        for (int d = 0; d < DS; d++) {
            sa[d] = group_sum(sa[d], 64);
            for (int o = 1; o < 64; o <<= 1) sm[d] = fmaxf(sm[d], __shfl_xor(sm[d], o));
        }
        if (lane == 0) {
#pragma unroll
            for (int d = 0; d < DS; d++) {
                wave_red[wave * DS + d] = sa[d];
                wave_mx[wave * DS + d] = sm[d];
            }
        }
        __syncthreads();
        if (tid < DS) {
            const int d = tid;
            float t = 0.f, mx = 0.f;
            for (int w = 0; w < kTableWaves; w++) {
                t += wave_red[w * DS + d];
                mx = fmaxf(mx, wave_mx[w * DS + d]);
            }
            dim_sum[d] = t;
            dim_max[d] = mx;
            int k = 0;
            if (t > 0.f) {
                // the fp32 sums are low by at most ~140 ulp-units relative (128 terms
                // per lane, 6 butterfly levels, 8 waves); the margin 1 + 2^-10 covers
                // it, so 2^k * (exact sum) < 2^30 and every bucket sum of rounded
                // values stays below 2^30 + n_src/2 < 2^31
                int ev;
                frexpf(t * (1.0f + 0x1p-10f), &ev);  // t (1 + 2^-10) < 2^ev
                k = 30 - ev;
            }
            scale_exp[d] = k;
        }
        __syncthreads();
    }
    // per-dim scales as wave-uniform exponents
    int kd[DS];
#pragma unroll
    for (int d = 0; d < DS; d++) kd[d] = __builtin_amdgcn_readfirstlane(scale_exp[d]);
    // with `hist`, per pass of hashes: the bucket counts of its hashes (in the tables'
    // LDS, before they are zeroed), the largest count c, and per dim the exponent k
    // with 2^k (1 + 2^-10) min(sum |v|, c max |v|) < 2^30.  Every bucket sum of a dim
    // is at most both bounds, so the argument of the sum bound holds as it is.
    auto count_scales = [&](int h0, int gcount) {
        uint32_t *cnt = reinterpret_cast<uint32_t *>(tab);  // [gcount][2^tau] (fits in the tables)
        const int nb = cmask + 1;
        for (int e = tid; e < gcount * nb; e += kTableThreads) cnt[e] = 0u;
        __syncthreads();
        // (key, hash) pairs in code order, eight per thread in flight; key = p / gcount
        // from a float reciprocal (p < 2^22, exact as a float; off by at most one,
        // corrected)
        const int npairs = static_cast<int>(a.n_src) * gcount;
        const uint16_t *hcodes = a.src_codes + b * a.n_src * a.m;
        // all of a row's hashes in this pass, m a multiple of 8 and the codes 16-byte
        // aligned: eight codes (one row's hashes 8v mod m .. +7) per 16-byte load
        const bool vec = gcount == a.m && (a.m & 7) == 0 && (reinterpret_cast<uintptr_t>(hcodes) & 15) == 0;
        const int nvec = vec ? npairs / 8 : 0;
        for (int v0 = tid; v0 < nvec; v0 += 8 * kTableThreads) {
            uint4 w[8];
#pragma unroll
            for (int u = 0; u < 8; u++) w[u] = reinterpret_cast<const uint4 *>(hcodes)[min(v0 + u * kTableThreads, nvec - 1)];
#pragma unroll
            for (int u = 0; u < 8; u++) {
                const int vi = v0 + u * kTableThreads;
                if (vi < nvec) {
                    const int hb = (8 * vi) % a.m;
                    const uint32_t ws[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
#pragma unroll
                    for (int e = 0; e < 8; e++)
                        atomicAdd(&cnt[(hb + e) * nb + ((ws[e >> 1] >> (16 * (e & 1))) & cmask)], 1u);
                }
            }
        }
        const float inv_g = 1.0f / static_cast<float>(gcount);
        for (int p0 = vec ? npairs : tid; p0 < npairs; p0 += 8 * kTableThreads) {
            uint32_t cc[8];
            int hq[8];
#pragma unroll
            for (int u = 0; u < 8; u++) {
                const int p = min(p0 + u * kTableThreads, npairs - 1);
                int key = static_cast<int>(static_cast<float>(p) * inv_g);
                if (key * gcount > p) key--;
                if ((key + 1) * gcount <= p) key++;
                hq[u] = p - key * gcount;
                cc[u] = hcodes[key * a.m + h0 + hq[u]];
            }
#pragma unroll
            for (int u = 0; u < 8; u++)
                if (p0 + u * kTableThreads < npairs) atomicAdd(&cnt[hq[u] * nb + (cc[u] & cmask)], 1u);
        }
        __syncthreads();
        uint32_t c = 0u;
        for (int e = tid; e < gcount * nb; e += kTableThreads) c = max(c, cnt[e]);
        for (int o = 1; o < 64; o <<= 1) c = max(c, static_cast<uint32_t>(__shfl_xor(static_cast<int>(c), o)));
        if (lane == 0) wave_cnt[wave] = c;
        __syncthreads();
        if (tid < DS) {
            const int d = tid;
            uint32_t cm = 0u;
            for (int w = 0; w < kTableWaves; w++) cm = max(cm, wave_cnt[w]);
            // (c <= 65536 is exact in fp32 and the product rounds once: the margin
            // 1 + 2^-10 covers it as it covers the rounding of the sums)
            const float bound = fminf(dim_sum[d], static_cast<float>(cm) * dim_max[d]);
            int k = 0;
            if (bound > 0.f) {
                int ev;
                frexpf(bound * (1.0f + 0x1p-10f), &ev);
                k = 30 - ev;
            }
            scale_exp[d] = k;
        }
        __syncthreads();  // (also: every count has been read before the tables are zeroed)
#pragma unroll
        for (int d = 0; d < DS; d++) kd[d] = __builtin_amdgcn_readfirstlane(scale_exp[d]);
    };

    // lane roles
    // hashes rounded up to a power of two: fixed by (DS, KM) for the one- and
    // two-key step forms (the host picks them exactly for those products), so their
    // lane roles below are compile-time constants
    constexpr int GPC = KM == 0 ? 2 * 64 / DS : (KM == 1 ? 64 / DS : 0);
    int GP = GPC;
    if constexpr (GPC == 0) {
        GP = 1;
        while (GP < G) GP <<= 1;
    }
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
    // gather lanes per query: 4 (8 for 64 hashes, so that a lane sums at most 8
    // hashes; fewer when there are fewer hashes)
    const int L = GP <= 4 ? GP : (GP / 8 > 4 ? GP / 8 : 4);
    const int HL = GP / L;                 // hashes per gather lane (<= 8)
    const int QPI = 64 / L;                // queries per gather instruction
    const int gq = lane / L, gr = lane % L;

    const int ngroups = (a.m + G - 1) / G;
    const int64_t src_row0 = b * a.n_src, dst_row0 = b * a.n_dst;
    const float inv_m = 1.0f / static_cast<float>(a.m);
    for (int grp = 0; grp < ngroups; grp++) {
        // no loads in flight from the previous group's gather (its last prefetches are
        // never used): otherwise the scatter below, whose registers they may occupy,
        // would wait for them on every chunk (vmcnt(0), all other counters untouched)
        __builtin_amdgcn_s_waitcnt(0x0F70);
        const int h0 = grp * G;
        const int gcount = min(G, a.m - h0);
        if (a.hist) count_scales(h0, gcount);
        {
            const int words = (cmask + 1) * G * P;  // even
            ulonglong2 *t2 = reinterpret_cast<ulonglong2 *>(tab);
            for (int e = tid; e < words / 2; e += kTableThreads) t2[e] = make_ulonglong2(0ull, 0ull);
        }
        __syncthreads();

        // ---- scatter
        // A wave owns 64-key chunks wave, wave+8, ...  Lane = key first loads and
        // quantises the chunk's values into the wave's staging area; then each step adds
        // one (KM 0) or two (KM 1) keys into the tables, every lane taking its (hash,
        // word) combo.  The words of eight steps are read from the staging area while the
        // previous eight steps' atomics issue; the codes a lane needs are fetched 32 steps
        // ahead and a chunk's values one chunk ahead, so no step waits for memory.
        if constexpr (KM < 2) {
            constexpr int KPI_C = KM == 0 ? 1 : 2;
            constexpr int SPC = 64 / KPI_C;  // steps per chunk
            constexpr int NG = SPC / 8;      // groups of eight steps per chunk
            const int64_t nchunks = (a.n_src + 63) / 64;
            const int mychunks = wave < nchunks ? static_cast<int>((nchunks - wave + kTableWaves - 1) / kTableWaves) : 0;
            const int hh = sh[0], pp = sp[0];
            const bool hok = hh < gcount;
            // codes are read as the aligned 32-bit pair holding the lane's code (m is even
            // and the codes 4-byte aligned for these forms), from a uniform per-head base
            // with 32-bit per-lane offsets (n*m < 2^22); the pair's half is a lane constant
            const uint32_t *cbase = reinterpret_cast<const uint32_t *>(a.src_codes + src_row0 * a.m);
            const int nsrc = static_cast<int>(a.n_src);
            const int tab_words = (cmask + 1) * G * P;
            // the lane's word is code * G * P + hh * P + pp: per step one bit-field extract
            // (the code) and one 24-bit multiply-add give its LDS byte address.  A lane
            // whose hash does not exist extracts a 0-bit code and adds into a private
            // dummy slot.  Keys past the end add zero words into real slots (their values
            // are zeroed, their codes read from a clamped row), so a step has no branch
            const uint32_t rowb = static_cast<uint32_t>(G * P) * 8u;
            const uint32_t loffb = static_cast<uint32_t>(hok ? hh * P + pp : tab_words + lane) * 8u;
            const uint32_t cwid = hok ? static_cast<uint32_t>(a.tau) : 0u;
            unsigned char *tabb = reinterpret_cast<unsigned char *>(tab);
            // codes are fetched kAhead steps ahead of their use, from a clamped (always
            // valid) row, into a ring of full registers (a 16-bit ring gets packed, and
            // packing at the chunk loop's back edge waits for every load in flight).  With
            // one key per step the row is the same for the whole wave: a uniform row
            // pointer and a per-lane constant offset, no per-lane address arithmetic
            constexpr int kAhead = 32;
            static_assert(SPC % kAhead == 0, "prefetch distance must divide the chunk");
            const uint32_t last = static_cast<uint32_t>(nsrc - 1), mm = static_cast<uint32_t>(a.m);
            const uint32_t hcol = static_cast<uint32_t>(h0) + (hok ? static_cast<uint32_t>(hh) : 0u);
            const uint32_t csh = (hcol & 1u) * 16u;
            const uint32_t hpair = hcol >> 1;  // the lane's 32-bit pair within a row (m even)
            auto code_at = [&](int tc, int st) -> uint32_t {
                const uint32_t row = static_cast<uint32_t>((wave + kTableWaves * tc) * 64 + st * KPI_C);
                if constexpr (KPI_C == 1)
                    return ld<uint32_t>(cbase + min(row, last) * (mm >> 1), hpair * 4u);
                else
                    return ld<uint32_t>(cbase, (__umul24(min(row + static_cast<uint32_t>(slot), last), mm >> 1) + hpair) * 4u);
            };
            // values of a chunk, lane = key, from a clamped row; rows past the end are
            // zeroed when the chunk is quantised (a select right after the load would
            // make the load wait)
            auto load_vals = [&](float v[DS], int tc) {
                const int j = (wave + kTableWaves * tc) * 64 + lane;
                load_slice<BF16, DS>(a.values, vbase + static_cast<int64_t>(min(j, nsrc - 1)) * D, v);
            };
            uint32_t cr[kAhead];
            float vr[DS];
            // this wave's staging area: the packed words of its chunk, [key][P]
            unsigned long long *wstage = tab + tab_words + 64 + wave * 64 * P;
            // (values before codes: at the top of the chunk loop the values are then
            // older than every code load in flight, on entry as on the back edge)
            if (mychunks > 0) {
                load_vals(vr, 0);
#pragma unroll
                for (int st = 0; st < kAhead; st++) cr[st] = code_at(0, st);
            }
            for (int tc = 0; tc < mychunks; tc++) {
                const bool kok = (wave + kTableWaves * tc) * 64 + lane < nsrc;
                // quantise and publish this chunk's words (lane = key), then start
                // fetching the next chunk's values (the last chunk fetches itself again)
#pragma unroll
                for (int p = 0; p < P; p++) {
                    const int lo = kok ? __float2int_rn(ldexpf(vr[2 * p], kd[2 * p])) : 0;
                    const int hi = kok ? __float2int_rn(ldexpf(vr[2 * p + 1], kd[2 * p + 1])) : 0;
                    wstage[lane * P + p] = (static_cast<unsigned long long>(static_cast<uint32_t>(hi)) << 32) +
                                           static_cast<unsigned long long>(static_cast<long long>(lo));
                }
                // the staging area is private to this wave and LDS executes a wave's
                // accesses in order: only the compiler must keep the reads below after
                // these writes (and the next chunk's writes after the reads)
                asm volatile("" ::: "memory");
                load_vals(vr, min(tc + 1, mychunks - 1));
                unsigned long long wd[2][8];
                auto read_words = [&](unsigned long long w[8], int g) {
#pragma unroll
                    for (int u = 0; u < 8; u++) w[u] = wstage[((8 * g + u) * KPI_C + slot) * P + pp];
                };
                read_words(wd[0], 0);
#pragma unroll
                for (int g = 0; g < NG; g++) {
                    if (g + 1 < NG) read_words(wd[(g + 1) & 1], g + 1);
#pragma unroll
                    for (int u = 0; u < 8; u++) {
                        const int st = 8 * g + u;
                        const uint32_t code = __builtin_amdgcn_ubfe(cr[st % kAhead], csh, cwid);
                        atomicAdd(reinterpret_cast<unsigned long long *>(tabb + __umul24(code, rowb) + loffb),
                                  wd[g & 1][u]);
                        cr[st % kAhead] = st + kAhead < SPC ? code_at(tc, st + kAhead) : code_at(tc + 1, st + kAhead - SPC);
                    }
                    // keep the scheduler from hoisting the unrolled chunk (register pressure)
                    __builtin_amdgcn_sched_barrier(0);
                }
                asm volatile("" ::: "memory");
            }
        } else {
            // general case (few hashes, wide slices): one step at a time, combos in NI passes
            for (int ii = 0; ii < NI; ii++) {
                const int hh = sh[ii], pp = sp[ii];
                const bool hok = hh < gcount;
                for (int64_t j0 = static_cast<int64_t>(wave) * 64; j0 < a.n_src;
                     j0 += static_cast<int64_t>(kTableWaves) * 64) {
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
                            const int lo = __float2int_rn(ldexpf(v[2 * p], kd[2 * p]));
                            const int hi = __float2int_rn(ldexpf(v[2 * p + 1], kd[2 * p + 1]));
                            const unsigned long long w =
                                (static_cast<unsigned long long>(static_cast<uint32_t>(hi)) << 32) +
                                static_cast<unsigned long long>(static_cast<long long>(lo));
                            pw[2 * p] = static_cast<uint32_t>(w);
                            pw[2 * p + 1] = static_cast<uint32_t>(w >> 32);
                        }
                    }
                    const int nk = static_cast<int>(a.n_src - j0 < 64 ? a.n_src - j0 : 64);
                    for (int kk = 0; kk < nk; kk += KPI) {
                        uint32_t w[2 * P];
#pragma unroll
                        for (int d = 0; d < 2 * P; d++) w[d] = __shfl(pw[d], (kk + slot) & 63);
                        const int key = kk + slot;
                        if (key < nk && hok) {
                            uint32_t lo = w[0], hi = w[1];
#pragma unroll
                            for (int p = 1; p < P; p++) {
                                lo = pp == p ? w[2 * p] : lo;
                                hi = pp == p ? w[2 * p + 1] : hi;
                            }
                            const int c = a.src_codes[(src_row0 + j0 + key) * a.m + h0 + hh] & cmask;
                            atomicAdd(&tab[(c * G + hh) * P + pp], (static_cast<unsigned long long>(hi) << 32) | lo);
                        }
                    }
                }
            }
        }
        __syncthreads();

        // ---- integer sums -> floats scaled by 2^-k_d / m, in place (a packed word and
        // its two floats have the same 8 bytes).  Word e holds dims 2p, 2p+1 with
        // p = e mod P, and P divides the thread count, so p is fixed per thread.
        {
            static_assert(kTableThreads % P == 0, "word slot must be fixed per thread");
            const int words = (cmask + 1) * G * P;
            const int pw = tid % P;
            int klo = kd[0], khi = kd[1];
#pragma unroll
            for (int p = 1; p < P; p++) {
                klo = pw == p ? kd[2 * p] : klo;
                khi = pw == p ? kd[2 * p + 1] : khi;
            }
            float2 *tf = reinterpret_cast<float2 *>(tab);
            for (int e = tid; e < words; e += kTableThreads) {
                int lo, hi;
                unpack(tab[e], lo, hi);
                tf[e] = make_float2(ldexpf(static_cast<float>(lo), -klo) * inv_m,
                                    ldexpf(static_cast<float>(hi), -khi) * inv_m);
            }
        }
        __syncthreads();

        // ---- gather: out[i][slice*DS + d] (+)= sum_h table[code_h(i)][h][d]
        // (the codes of the wave's next few query groups are fetched ahead)
        // (the single-pass and multi-pass output paths are separate instantiations:
        // sharing blocks with the accumulator loads of the multi-pass path would make
        // every single-pass store wait for all outstanding loads)
        auto gather = [&](auto single) {
            constexpr bool SINGLE = decltype(single)::value;
        {
            int hh[8];
#pragma unroll
            for (int t = 0; t < 8; t++) hh[t] = gr + L * ((t + gq) % (HL > 0 ? HL : 1));
            // codes of a query group: loads from clamped (always valid) positions,
            // validity applied afterwards, so the loads stay in flight
            // (raw codes only: a per-lane select on a loaded value makes the compiler
            // branch around the load and wait for it; validity is kept apart.  The one-
            // and two-key forms read the aligned 32-bit pair holding the code, so that the
            // ring of codes in flight needs no widening copy at the loop's back edge)
            const uint32_t qlast = static_cast<uint32_t>(a.n_dst - 1), mm = static_cast<uint32_t>(a.m);
            uint32_t hcol[8], csh[8];
#pragma unroll
            for (int t = 0; t < 8; t++) {
                hcol[t] = static_cast<uint32_t>(h0) + (hh[t] < gcount ? static_cast<uint32_t>(hh[t]) : 0u);
                csh[t] = KM < 2 ? (hcol[t] & 1u) * 16u : 0u;
            }
            const uint16_t *qhead = a.dst_codes + dst_row0 * a.m;
            // the byte offset of the 32-bit pair holding hash t's code within a row (m even)
            uint32_t hbyte[8];
#pragma unroll
            for (int t = 0; t < 8; t++) hbyte[t] = (hcol[t] >> 1) * 4u;
            auto fetch = [&](uint32_t cc[8], int64_t i0) {
                const int64_t i = i0 + gq;
                const uint32_t icl = i < a.n_dst ? static_cast<uint32_t>(i) : qlast;
                const uint32_t qbyte = __umul24(icl, 2u * mm);  // the query's row of codes
#pragma unroll
                for (int t = 0; t < 8; t++) {
                    if (t < HL) {
                        if constexpr (KM < 2)
                            cc[t] = ld<uint32_t>(qhead, qbyte + hbyte[t]);
                        else
                            cc[t] = qhead[icl * mm + hcol[t]];
                    }
                }
            };
            // weight of hash t's row: 1 where the lane's hash t exists.  A query past the
            // end reads clamped, valid rows and is never stored, so it needs no weight
            float wt[8];
#pragma unroll
            for (int t = 0; t < 8; t++) wt[t] = (t < HL && hh[t] < gcount) ? 1.f : 0.f;
            // byte offset of hash t's row within a bucket's block of G rows, and of one bucket
            uint32_t hrow[8];
#pragma unroll
            for (int t = 0; t < 8; t++) hrow[t] = static_cast<uint32_t>(min(hh[t], gcount - 1)) * (DS * 4u);
            const uint32_t bucket_bytes = static_cast<uint32_t>(G) * (DS * 4u);
            const unsigned char *tabc = reinterpret_cast<const unsigned char *>(tab);
            const int64_t step = static_cast<int64_t>(kTableWaves) * QPI;
            // codes of the next kGD query groups are in flight while one is summed
            constexpr int kGD = KM < 2 ? 4 : 2;
            uint32_t cR[kGD][8];
            // (issued in ring order, which the first groups' waits assume)
#pragma unroll
            for (int u = 0; u < kGD; u++) {
                fetch(cR[u], static_cast<int64_t>(wave) * QPI + u * step);
                __builtin_amdgcn_sched_barrier(0);
            }
            for (int64_t ib = static_cast<int64_t>(wave) * QPI; ib < a.n_dst; ib += kGD * step) {
#pragma unroll
                for (int u = 0; u < kGD; u++) {
                    const int64_t i0 = ib + u * step;
                    if (i0 >= a.n_dst) break;
                    const int64_t i = i0 + gq;
                    const bool qok = i < a.n_dst;
                    // every lane reads a row (a lane whose hash does not exist reads a
                    // clamped row and weights it by 0): no divergent branch between the
                    // reads, and all of a group's reads are issued before the first is used
                    float xs[8][DS];
#pragma unroll
                    for (int t = 0; t < 8; t++) {
                        if (t < HL) {
                            // (a 24-bit multiply: a 32-bit one becomes v_mad_u64_u32, whose unused
                            // high addend half can be allocated to a load in flight, which then
                            // has to be waited for)
                            const uint32_t code = __builtin_amdgcn_ubfe(cR[u][t], csh[t], static_cast<uint32_t>(a.tau));
                            const float *row = reinterpret_cast<const float *>(tabc + __umul24(code, bucket_bytes) + hrow[t]);
                            if constexpr (DS == 2) {
                                const float2 x = *reinterpret_cast<const float2 *>(row);
                                xs[t][0] = x.x;
                                xs[t][1] = x.y;
                            } else {
#pragma unroll
                                for (int d = 0; d < DS; d += 4) {
                                    const float4 x = *reinterpret_cast<const float4 *>(row + d);
                                    xs[t][d] = x.x;
                                    xs[t][d + 1] = x.y;
                                    xs[t][d + 2] = x.z;
                                    xs[t][d + 3] = x.w;
                                }
                            }
                        }
                    }
                    fetch(cR[u], i0 + kGD * step);
                    float acc[DS];
#pragma unroll
                    for (int d = 0; d < DS; d++) acc[d] = 0.f;
#pragma unroll
                    for (int t = 0; t < 8; t++) {
                        if (t < HL) {
#pragma unroll
                            for (int d = 0; d < DS; d++) acc[d] = fmaf(xs[t][d], wt[t], acc[d]);
                        }
                    }
                    // every lane of the query's group holds the sums; lane c4 % L
                    // stores dims [4 c4, 4 c4 + 4) (or the two dims of a 2-wide slice)
#pragma unroll
                    for (int d = 0; d < DS; d++) acc[d] = group_sum(acc[d], L);
                    if (qok) {
                        const int64_t obase = (dst_row0 + i) * D + slice * DS;
                        constexpr int CW = DS < 4 ? DS : 4;
#pragma unroll
                        for (int c4 = 0; c4 < DS / CW; c4++) {
                            if (gr != c4 % L) continue;
                            float v[CW];
#pragma unroll
                            for (int e = 0; e < CW; e++) v[e] = acc[c4 * CW + e];
                            const int64_t o = obase + c4 * CW;
                            if constexpr (!SINGLE) {
                                // the same lane owns this chunk in every group
                                if (grp > 0) {
                                    if constexpr (CW == 4) {
                                        const float4 pv = *reinterpret_cast<const float4 *>(a.acc + o);
                                        v[0] += pv.x; v[1] += pv.y; v[2] += pv.z; v[3] += pv.w;
                                    } else {
                                        const float2 pv = *reinterpret_cast<const float2 *>(a.acc + o);
                                        v[0] += pv.x; v[1] += pv.y;
                                    }
                                }
                            }
                            if (SINGLE || grp == ngroups - 1) {
                                if constexpr (BF16) {
                                    if constexpr (CW == 4) {
                                        uint2 w2;
                                        w2.x = static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
                                        w2.y = static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
                                        *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(a.out) + o) = w2;
                                    } else {
                                        *reinterpret_cast<uint32_t *>(static_cast<uint16_t *>(a.out) + o) =
                                            static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
                                    }
                                    continue;
                                }
                            }
                            // fp32 output, or the fp32 running sums of a multi-pass bf16 run
                            float *dst = (BF16 || !(SINGLE || grp == ngroups - 1)) ? a.acc : static_cast<float *>(a.out);
                            if constexpr (CW == 4)
                                *reinterpret_cast<float4 *>(dst + o) = make_float4(v[0], v[1], v[2], v[3]);
                            else
                                *reinterpret_cast<float2 *>(dst + o) = make_float2(v[0], v[1]);
                        }
                    }
                }
            }
        }
        };
        if (ngroups == 1)
            gather(std::true_type{});
        else
            gather(std::false_type{});
        __syncthreads();
    }
}

template <bool BF16, int DS>
void launch_table_km(int km, const TableArgs &a, size_t lds, hipStream_t stream) {
    const int64_t blocks = a.bh * (D / DS);
    const dim3 grid(static_cast<unsigned>(blocks)), block(kTableThreads);
    if (km == 0)
        hipLaunchKernelGGL((table_kernel<BF16, DS, 0>), grid, block, lds, stream, a);
    else if (km == 1)
        hipLaunchKernelGGL((table_kernel<BF16, DS, 1>), grid, block, lds, stream, a);
    else
        hipLaunchKernelGGL((table_kernel<BF16, DS, 2>), grid, block, lds, stream, a);
}

// Step form of a table launch: 0 -> one key per step, 1 -> two keys per step (both
// with LDS staging of a chunk's packed words), 2 -> the general form.
int table_step_form(const TableArgs &a, int ds) {
    int gp = 1;
    while (gp < a.G) gp <<= 1;
    const int cpk = gp * (ds / 2);
    // the one- and two-key forms read codes as aligned 32-bit pairs
    const bool pairs = a.m % 2 == 0 && (reinterpret_cast<uintptr_t>(a.src_codes) & 3) == 0 &&
                       (reinterpret_cast<uintptr_t>(a.dst_codes) & 3) == 0;
    return (ds > 8 || !pairs) ? 2 : (cpk == 64 ? 0 : (cpk == 32 ? 1 : 2));
}

template <bool BF16>
hipError_t launch_table_ds(int ds, int km, const TableArgs &a, size_t lds, hipStream_t stream) {
    KernelTimer timer("table_kernel", stream);
    switch (ds) {
        case 2: launch_table_km<BF16, 2>(km, a, lds, stream); break;
        case 4: launch_table_km<BF16, 4>(km, a, lds, stream); break;
        case 8: launch_table_km<BF16, 8>(km, a, lds, stream); break;
        case 16: launch_table_km<BF16, 16>(km, a, lds, stream); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
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
    TablePlan p = plan_table(m, tau);
    // a head or two: narrower slices, so that more workgroups share the work (one head
    // of 512 rows: 16 -> 32 workgroups, 15 -> 11.6 us); the hashes per pass stay
    while (p.DS > 2 && bh * (D / p.DS) < kTableFewBlocks) {
        p.DS /= 2;
        p.lds /= 2;
    }
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
    // fp32 outputs of long sequences: the sum bound grows with n_src (its rounding
    // step with it), the largest bucket count does not
    a.hist = !bf16 && n_src > kTableHistRows ? 1 : 0;
    // the one- and two-key step forms also need one private dummy word per lane
    // (targets of lanes without a valid key) and per-wave staging of a chunk's
    // packed words (64 keys x DS/2 words); the general form needs neither (with 128
    // KiB of tables and 16-dim slices they would not fit beside them)
    const int km = table_step_form(a, p.DS);
    const size_t lds = p.lds + (km < 2 ? 64 * sizeof(unsigned long long) +
                                             static_cast<size_t>(kTableWaves) * 64 * (p.DS / 2) *
                                                 sizeof(unsigned long long)
                                       : 0);
    return bf16 ? launch_table_ds<true>(p.DS, km, a, lds, stream) : launch_table_ds<false>(p.DS, km, a, lds, stream);
}

}  // namespace yoso
