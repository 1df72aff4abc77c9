// Microbenchmarks and lane-layout checks of the gfx950 facts the YOSO kernels are designed around.
//
//   hw_facts            every rate below, then the two checks; prints a markdown table
//   hw_facts --checks   the two checks only (the GPU test runs this)
//
// Checks (the exit status is 1 if one fails):
//   * fp16 subnormal inputs of v_mfma_f32_16x16x32_f16 are multiplied exactly, not flushed to zero
//     (the fp16 hi/lo splits of the backward rely on it for small low parts);
//   * ds_read_b64_tr_b16 hands destination lane 4a+b of each 16-lane group element b of the 8 bytes
//     addressed by source lane 4i+a of that group, as element i (the pair kernel's transposed reads).
//
// Rates are per compute unit and clock where the unit is the CU (the clock is taken as 2.4 GHz, not
// measured), else whole-chip bytes or flops per second. Every access stays inside its buffer: LDS
// indexes are masked to the array size and global offsets are reduced modulo the row count.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#define CK(x)                                                                              \
  do {                                                                                     \
    hipError_t e_ = (x);                                                                   \
    if (e_ != hipSuccess) {                                                                \
      std::fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
      std::exit(2);                                                                        \
    }                                                                                      \
  } while (0)

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef short short4v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) short4v lds_short4;

static constexpr double kClock = 2.4e9;

__device__ __forceinline__ uint32_t lcg(uint32_t s) { return s * 1664525u + 1013904223u; }

// ---- LDS atomics: 1024 threads, a 128 KiB table, one atomic per lane per iteration.
template <class T, bool RANDOM>
__global__ __launch_bounds__(1024) void lds_atom_kernel(T *out, int iters) {
  constexpr int N = 131072 / sizeof(T);
  __shared__ T tab[N];
  for (int i = threadIdx.x; i < N; i += 1024) tab[i] = T(0);
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t s = lcg(blockIdx.x * 1024u + threadIdx.x);
  for (int it = 0; it < iters; it++) {
    int a;
    if (RANDOM) {
      s = lcg(s);
      a = (s >> 8) & (N - 1);
    } else {
      a = ((it * 16 + wave) * 64 + lane) & (N - 1);
    }
    atomicAdd(&tab[a], T(1));
  }
  __syncthreads();
  T acc = T(0);
  for (int i = threadIdx.x; i < N; i += 1024) acc += tab[i];
  out[blockIdx.x * 1024 + threadIdx.x] = acc;
}

// ---- LDS contiguous reads or writes of W bytes per lane; each wave owns 8 KiB.
template <int W, bool WRITE>
__global__ __launch_bounds__(256) void lds_rw_kernel(float *out, int iters) {
  __shared__ __align__(16) unsigned char lds[4 * 8192];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned char *t = lds + wave * 8192;
  for (int i = threadIdx.x; i < 4 * 8192 / 16; i += 256) reinterpret_cast<uint4 *>(lds)[i] = make_uint4(i, i, i, i);
  __syncthreads();
  float acc = 0.f;
  unsigned v = lane;
  constexpr int PER_PASS = 8192 / (64 * W);
  for (int it = 0; it < iters; it++) {
#pragma unroll
    for (int i = 0; i < PER_PASS; i++) {
      unsigned char *p = t + i * 64 * W + lane * W;
      if (WRITE) {
        if (W == 4) *reinterpret_cast<unsigned *>(p) = v;
        if (W == 8) *reinterpret_cast<uint2 *>(p) = make_uint2(v, v);
        if (W == 16) *reinterpret_cast<uint4 *>(p) = make_uint4(v, v, v, v);
      } else {
        if (W == 4) acc += __uint_as_float(*reinterpret_cast<const unsigned *>(p));
        if (W == 8) {
          const uint2 a = *reinterpret_cast<const uint2 *>(p);
          acc += __uint_as_float(a.x) * __uint_as_float(a.y);
        }
        if (W == 16) {
          const uint4 a = *reinterpret_cast<const uint4 *>(p);
          acc += __uint_as_float(a.x) * __uint_as_float(a.y) + __uint_as_float(a.z) * __uint_as_float(a.w);
        }
      }
    }
    v += 1;
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): one pass completes before the next is issued
  }
  __syncthreads();
  out[blockIdx.x * 256 + threadIdx.x] = acc + __uint_as_float(reinterpret_cast<const unsigned *>(lds)[threadIdx.x]);
}

// ---- L2 -> CU: each quarter-wave reads one 256-byte row of a 2 MiB set (8192 rows), rows drawn at random.
__global__ __launch_bounds__(256) void l2_read_kernel(const uint4 *buf, uint32_t *out, int iters) {
  const int lane = threadIdx.x & 63;
  uint32_t s = lcg(blockIdx.x * 256u + (threadIdx.x & ~15u));
  uint32_t acc = 0;
  for (int it = 0; it < iters; it++) {
    s = lcg(s);
    const uint32_t row = (s >> 8) & 8191u;
    const uint4 x = buf[row * 16u + (lane & 15)];
    acc ^= x.x ^ x.y ^ x.z ^ x.w;
  }
  out[blockIdx.x * 256 + threadIdx.x] = acc;
}

// ---- HBM streaming read: grid-stride over n16 16-byte words.
__global__ __launch_bounds__(256) void hbm_read_kernel(const uint4 *buf, int64_t n16, uint32_t *out) {
  uint32_t acc = 0;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n16; i += stride) {
    const uint4 x = buf[i];
    acc ^= x.x ^ x.y ^ x.z ^ x.w;
  }
  out[blockIdx.x * 256 + threadIdx.x] = acc;
}

// ---- global fp32 atomics into [rows][64]: each wave adds to one random 256-byte row per iteration.
__global__ __launch_bounds__(256) void global_atomic_kernel(float *buf, uint32_t rows, int iters) {
  const int lane = threadIdx.x & 63;
  uint32_t s = lcg(blockIdx.x * 4u + (threadIdx.x >> 6));
  for (int it = 0; it < iters; it++) {
    s = lcg(s);
    const int64_t off = static_cast<int64_t>((s >> 4) % rows) * 64 + lane;
    unsafeAtomicAdd(buf + off, 1.0f);
  }
}

// ---- MFMA issue rate: each wave runs ACC independent accumulator chains of one instruction shape.
typedef float floatx16 __attribute__((ext_vector_type(16)));
template <int ACC>
__global__ __launch_bounds__(256) void mfma32_kernel(float *out, int iters, float seed) {
  floatx16 acc[ACC];
  for (int i = 0; i < ACC; i++)
    for (int j = 0; j < 16; j++) acc[i][j] = 0.f;
  half8 a8, b8;
  for (int i = 0; i < 8; i++) {
    a8[i] = static_cast<_Float16>(seed * (threadIdx.x + i));
    b8[i] = static_cast<_Float16>(seed * i);
  }
  for (int it = 0; it < iters; it++) {
#pragma unroll
    for (int i = 0; i < ACC; i++) acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a8, b8, acc[i], 0, 0, 0);
  }
  float s = 0.f;
  for (int i = 0; i < ACC; i++)
    for (int j = 0; j < 16; j++) s += acc[i][j];
  out[blockIdx.x * 256 + threadIdx.x] = s;
}

template <bool K32, int ACC>
__global__ __launch_bounds__(256) void mfma_kernel(float *out, int iters, float seed) {
  floatx4 acc[ACC];
  for (int i = 0; i < ACC; i++) acc[i] = floatx4{0, 0, 0, 0};
  half8 a8, b8;
  half4 a4, b4;
  for (int i = 0; i < 8; i++) {
    a8[i] = static_cast<_Float16>(seed * (threadIdx.x + i));
    b8[i] = static_cast<_Float16>(seed * i);
  }
  for (int i = 0; i < 4; i++) {
    a4[i] = a8[i];
    b4[i] = b8[i];
  }
  for (int it = 0; it < iters; it++) {
#pragma unroll
    for (int i = 0; i < ACC; i++) {
      if constexpr (K32)
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a8, b8, acc[i], 0, 0, 0);
      else
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x16f16(a4, b4, acc[i], 0, 0, 0);
    }
  }
  float s = 0.f;
  for (int i = 0; i < ACC; i++) s += acc[i][0] + acc[i][1] + acc[i][2] + acc[i][3];
  out[blockIdx.x * 256 + threadIdx.x] = s;
}

// ---- check: one wave, every A element a, every B element b; each output is the exact 32*a*b.
__global__ __launch_bounds__(64) void subnormal_kernel(float *out, float a, float b) {
  half8 av, bv;
  for (int i = 0; i < 8; i++) {
    av[i] = static_cast<_Float16>(a);
    bv[i] = static_cast<_Float16>(b);
  }
  const floatx4 r = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bv, floatx4{0, 0, 0, 0}, 0, 0, 0);
  for (int j = 0; j < 4; j++) out[threadIdx.x * 4 + j] = r[j];
}

// ---- check: LDS holds lds[i] = i; three address patterns, each lane's address 8-byte aligned and in bounds.
__device__ __host__ inline int tr_addr(int pattern, int lane) {
  if (pattern == 0) return lane * 4;
  if (pattern == 1) return lane * 64;
  return (lane % 16) * 64 + (lane / 16) * 4;
}

__global__ __launch_bounds__(64) void tr_kernel(short *out) {
  __shared__ __align__(16) short lds[4096];
  for (int i = threadIdx.x; i < 4096; i += 64) lds[i] = static_cast<short>(i);
  __syncthreads();
  const int l = threadIdx.x;
  for (int p = 0; p < 3; p++) {
    const short4v r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4 *)(lds + tr_addr(p, l)));
    for (int i = 0; i < 4; i++) out[(p * 64 + l) * 4 + i] = r[i];
  }
}

// ---------------------------------------------------------------------------------------------------------
struct Timer {
  hipEvent_t a, b;
  Timer() {
    CK(hipEventCreate(&a));
    CK(hipEventCreate(&b));
  }
  ~Timer() {
    (void)hipEventDestroy(a);
    (void)hipEventDestroy(b);
  }
  template <class F>
  double ms(F launch) {  // one untimed launch, then the best of three timed ones
    launch();
    CK(hipGetLastError());
    CK(hipDeviceSynchronize());
    double best = 1e30;
    for (int r = 0; r < 3; r++) {
      CK(hipEventRecord(a));
      launch();
      CK(hipEventRecord(b));
      CK(hipEventSynchronize(b));
      float t;
      CK(hipEventElapsedTime(&t, a, b));
      best = t < best ? t : best;
    }
    return best;
  }
};

static int g_cus = 256;
static void row(const char *what, double value, const char *unit) { std::printf("| %s | %.3g %s |\n", what, value, unit); }

template <class T, bool RANDOM>
static void lds_atom_rate(void *scratch, const char *name) {
  const int blocks = g_cus * 4, iters = 2048;
  Timer t;
  const double ms = t.ms([&] { lds_atom_kernel<T, RANDOM><<<blocks, 1024>>>(static_cast<T *>(scratch), iters); });
  row(name, double(blocks) * 1024 * iters / (ms * 1e-3) / kClock / g_cus, "lane-ops/clk/CU");
}

template <int W, bool WRITE>
static void lds_rw(float *scratch, const char *name) {
  const int blocks = 1024, iters = 400;
  Timer t;
  const double ms = t.ms([&] { lds_rw_kernel<W, WRITE><<<blocks, 256>>>(scratch, iters); });
  row(name, double(blocks) * 4 * iters * 8192 / (ms * 1e-3) / kClock / g_cus, "B/clk/CU");
}

template <bool K32>
static void mfma(float *scratch, const char *name) {
  const int blocks = 2048, iters = 4096;
  constexpr int ACC = 8;
  Timer t;
  const double ms = t.ms([&] { mfma_kernel<K32, ACC><<<blocks, 256>>>(scratch, iters, 1e-3f); });
  const double flops = 2.0 * 16 * 16 * (K32 ? 32 : 16) * ACC * iters * (blocks * 4.0);
  const double clk_per_instr = ms * 1e-3 * kClock / (double(ACC) * iters * blocks * 4 / (4.0 * g_cus));
  std::printf("| %s, %d independent accumulators per wave | %.3g PFLOP/s, %.1f clk per instruction per SIMD |\n", name, ACC,
              flops / (ms * 1e-3) / 1e15, clk_per_instr);
}

static void mfma32(float *scratch) {
  const int blocks = 2048, iters = 2048;
  constexpr int ACC = 4;
  Timer t;
  const double ms = t.ms([&] { mfma32_kernel<ACC><<<blocks, 256>>>(scratch, iters, 1e-3f); });
  const double flops = 2.0 * 32 * 32 * 16 * ACC * iters * (blocks * 4.0);
  const double clk_per_instr = ms * 1e-3 * kClock / (double(ACC) * iters * blocks * 4 / (4.0 * g_cus));
  std::printf("| `v_mfma_f32_32x32x16_f16`, %d independent accumulators per wave | %.3g PFLOP/s, %.1f clk per instruction per SIMD |\n",
              ACC, flops / (ms * 1e-3) / 1e15, clk_per_instr);
}

static bool check_subnormals() {
  float *d;
  CK(hipMalloc(&d, 64 * 4 * sizeof(float)));
  // (a, b): a fp16 subnormal times a normal, and the smallest fp16 subnormal times a small normal
  const float cases[][2] = {{0x1p-20f, 1.0f}, {0x1p-24f, 0x1p-4f}, {0x1p-15f, 0x1p-10f}};
  bool ok = true;
  for (const auto &c : cases) {
    subnormal_kernel<<<1, 64>>>(d, c[0], c[1]);
    CK(hipGetLastError());
    float h[256];
    CK(hipMemcpy(h, d, sizeof h, hipMemcpyDeviceToHost));
    const float want = 32.0f * c[0] * c[1];
    for (float x : h) ok &= (x == want);
    std::printf("  mfma 16x16x32 f16: 32 * %a * %a = %a (exact %a)\n", c[0], c[1], h[0], want);
  }
  CK(hipFree(d));
  return ok;
}

static bool check_transpose_read() {
  short *d;
  CK(hipMalloc(&d, 3 * 64 * 4 * sizeof(short)));
  tr_kernel<<<1, 64>>>(d);
  CK(hipGetLastError());
  short h[3 * 64 * 4];
  CK(hipMemcpy(h, d, sizeof h, hipMemcpyDeviceToHost));
  CK(hipFree(d));
  bool ok = true;
  for (int p = 0; p < 3; p++)
    for (int L = 0; L < 64; L++) {
      const int g = L / 16, a = (L % 16) / 4, b = L % 4;
      for (int i = 0; i < 4; i++) ok &= h[(p * 64 + L) * 4 + i] == tr_addr(p, 16 * g + 4 * i + a) + b;
    }
  return ok;
}

int main(int argc, char **argv) {
  const bool checks_only = argc > 1 && std::strcmp(argv[1], "--checks") == 0;
  hipDeviceProp_t prop;
  CK(hipGetDeviceProperties(&prop, 0));
  g_cus = prop.multiProcessorCount;
  std::printf("device %s, %d compute units, clock taken as %.1f GHz\n\n", prop.gcnArchName, g_cus, kClock / 1e9);

  if (!checks_only) {
    const size_t scratch_bytes = size_t(4096) * 1024 * 8;  // large enough for every kernel's `out`
    void *scratch;
    CK(hipMalloc(&scratch, scratch_bytes));
    std::printf("| operation | measured |\n|---|---|\n");
    lds_atom_rate<float, false>(scratch, "LDS `ds_add_f32`, conflict-free");
    lds_atom_rate<float, true>(scratch, "LDS `ds_add_f32`, random");
    lds_atom_rate<uint32_t, false>(scratch, "LDS `ds_add_u32`, conflict-free");
    lds_atom_rate<uint32_t, true>(scratch, "LDS `ds_add_u32`, random");
    lds_atom_rate<unsigned long long, false>(scratch, "LDS `ds_add_u64`, conflict-free");
    lds_atom_rate<unsigned long long, true>(scratch, "LDS `ds_add_u64`, random");
    lds_rw<16, false>(static_cast<float *>(scratch), "LDS contiguous reads, 16 B per lane");
    lds_rw<8, false>(static_cast<float *>(scratch), "LDS contiguous reads, 8 B per lane");
    lds_rw<4, false>(static_cast<float *>(scratch), "LDS contiguous reads, 4 B per lane");
    lds_rw<16, true>(static_cast<float *>(scratch), "LDS contiguous writes, 16 B per lane");
    lds_rw<8, true>(static_cast<float *>(scratch), "LDS contiguous writes, 8 B per lane");
    lds_rw<4, true>(static_cast<float *>(scratch), "LDS contiguous writes, 4 B per lane");

    uint4 *set;
    CK(hipMalloc(&set, size_t(2) << 20));
    CK(hipMemset(set, 1, size_t(2) << 20));
    {
      const int blocks = 4096, iters = 512;
      Timer t;
      const double ms = t.ms([&] { l2_read_kernel<<<blocks, 256>>>(set, static_cast<uint32_t *>(scratch), iters); });
      row("L2 -> CU, random 256-byte rows of a 2 MiB set", double(blocks) * 16 * iters * 256 / (ms * 1e-3) / 1e12, "TB/s");
    }
    CK(hipFree(set));

    const size_t big = size_t(1) << 30;
    uint4 *hbm;
    CK(hipMalloc(&hbm, big));
    CK(hipMemset(hbm, 3, big));
    {
      const int blocks = g_cus * 16;
      Timer t;
      const double ms = t.ms([&] {
        hbm_read_kernel<<<blocks, 256>>>(hbm, int64_t(big / 16), static_cast<uint32_t *>(scratch));
      });
      row("HBM streaming read, 1 GiB", double(big) / (ms * 1e-3) / 1e12, "TB/s");
    }
    {
      const uint32_t rows = 1u << 16;  // 16 MiB of fp32 inside the 1 GiB buffer
      const int blocks = g_cus * 8, iters = 1024;
      Timer t;
      const double ms = t.ms([&] { global_atomic_kernel<<<blocks, 256>>>(reinterpret_cast<float *>(hbm), rows, iters); });
      row("global fp32 atomic adds, random rows of a 16 MiB buffer", double(blocks) * 256 * iters / (ms * 1e-3) / 1e9,
          "G floats/s");
    }
    CK(hipFree(hbm));

    mfma<true>(static_cast<float *>(scratch), "`v_mfma_f32_16x16x32_f16`");
    mfma<false>(static_cast<float *>(scratch), "`v_mfma_f32_16x16x16_f16`");
    mfma32(static_cast<float *>(scratch));
    CK(hipFree(scratch));
    std::printf("\n");
  }

  const bool sub = check_subnormals();
  const bool tr = check_transpose_read();
  std::printf("check fp16 subnormal products exact in MFMA: %s\n", sub ? "yes" : "NO");
  std::printf("check ds_read_b64_tr_b16 lane layout as documented: %s\n", tr ? "yes" : "NO");
  return sub && tr ? 0 : 1;
}
