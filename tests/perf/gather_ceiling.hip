// Measurement probe: throughput of dependent random reads on one GPU, by
// working-set size, record width, cache-policy bits and memory kind, plus a
// plain streaming copy. It explains the walk kernel's ceiling: a walk hop is
// one dependent random read that almost always misses L2.
//
// A second table separates the possible limits: the same cache lines spread
// over a larger address range (more pages, same cache footprint) tests TLB
// reach; several independent chains per lane and fewer lanes test whether the
// rate is set by the number of reads in flight.
//
// Every index is reduced modulo the table size, so all accesses are in bounds.
// Fine-grained and uncached allocations are never freed (the process ends).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

#define CK(x)                                                                      \
  do {                                                                             \
    hipError_t e_ = (x);                                                           \
    if (e_ != hipSuccess) {                                                        \
      std::printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);   \
      return 1;                                                                    \
    }                                                                              \
  } while (0)

typedef int32_t v2i __attribute__((ext_vector_type(2)));
typedef int32_t v4i __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t mix(uint32_t x) {
  x ^= x >> 16; x *= 0x7feb352dU; x ^= x >> 15; x *= 0x846ca68bU; x ^= x >> 16;
  return x;
}

// t[i].x = a pseudo-random index in [0, n)
__global__ void fill(v4i *t, uint64_t n) {
  for (uint64_t i = blockIdx.x * uint64_t(blockDim.x) + threadIdx.x; i < n; i += uint64_t(gridDim.x) * blockDim.x) {
    const uint32_t h = mix(uint32_t(i) * 2654435761u + 12345u);
    t[i] = v4i{int32_t((uint64_t(h) * n) >> 32), int32_t(h), int32_t(i), 0};
  }
}

// MODE 0: 8-byte loads (stride 16 B); 1: 16-byte loads; 2: 8-byte non-temporal
// loads; 3: 8-byte buffer loads with sc0 sc1 set.
template <int MODE>
__global__ __launch_bounds__(256) void chase(const v4i *__restrict__ t, uint64_t n, int steps, uint32_t *out) {
  const uint32_t lane = blockIdx.x * 256 + threadIdx.x;
  uint32_t idx = uint32_t((uint64_t(mix(lane)) * n) >> 32);
  uint32_t acc = 0;
  __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc((void *)t, 0, 0x7fffffff, 0x00020000);
  for (int s = 0; s < steps; ++s) {
    if (MODE == 1) {
      const v4i v = t[idx];
      idx = uint32_t(v.x); acc += uint32_t(v.y + v.z);
    } else {
      const v2i *p = reinterpret_cast<const v2i *>(t + idx);
      v2i v;
      if (MODE == 0) v = *p;
      else if (MODE == 2) v = __builtin_nontemporal_load(p);
      else v = __builtin_amdgcn_raw_buffer_load_b64(r, idx * 16u, 0, 17);
      idx = uint32_t(v.x); acc += uint32_t(v.y);
    }
  }
  out[lane] = acc + idx;
}

// Physical record of logical record i when the table's 128-byte lines (8
// records) are spread by a power-of-two factor g: line L lands at a pseudo-random
// line inside [L*g, L*g + g), so cache sets and channels stay uniformly used.
// The largest index is n*g - 1 for n a multiple of 8.
__device__ __forceinline__ uint64_t spread_index(uint32_t i, uint32_t g) {
  const uint64_t line = i >> 3;
  return ((line * g + (mix(uint32_t(line) ^ 0x5bd1e995u) & (g - 1))) << 3) | (i & 7u);
}

__global__ void fill_spread(v4i *t, uint32_t n, uint32_t g) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    const uint32_t h = mix(i * 2654435761u + 12345u);
    t[spread_index(i, g)] = v4i{int32_t((uint64_t(h) * n) >> 32), int32_t(h), int32_t(i), 0};
  }
}

// K independent chains per lane over a spread table, 16-byte reads.
template <int K>
__global__ __launch_bounds__(256) void chase_chains(const v4i *__restrict__ t, uint32_t n, uint32_t g, int steps,
                                                    uint32_t *out) {
  const uint32_t lane = blockIdx.x * 256 + threadIdx.x;
  uint32_t idx[K];
  uint32_t acc = 0;
#pragma unroll
  for (int k = 0; k < K; ++k) idx[k] = uint32_t((uint64_t(mix(lane * K + k)) * n) >> 32);
  for (int s = 0; s < steps; ++s) {
    v4i v[K];
#pragma unroll
    for (int k = 0; k < K; ++k) v[k] = t[spread_index(idx[k], g)];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      idx[k] = uint32_t(v[k].x);
      acc += uint32_t(v[k].y + v[k].z);
    }
  }
  uint32_t r = acc;
#pragma unroll
  for (int k = 0; k < K; ++k) r += idx[k];
  out[lane] = r;
}

__global__ void copy16(const v4i *a, v4i *b, uint64_t n) {
  for (uint64_t i = blockIdx.x * uint64_t(blockDim.x) + threadIdx.x; i < n; i += uint64_t(gridDim.x) * blockDim.x)
    b[i] = a[i];
}

static uint32_t host_out[1u << 21];

template <int MODE>
int run(const v4i *t, uint64_t n, uint32_t *out, const char *what, hipEvent_t a, hipEvent_t b) {
  const uint32_t lanes = 1u << 21;
  const int steps = 32;
  chase<MODE><<<lanes / 256, 256>>>(t, n, steps, out);
  CK(hipDeviceSynchronize());
  CK(hipEventRecord(a));
  chase<MODE><<<lanes / 256, 256>>>(t, n, steps, out);
  CK(hipEventRecord(b));
  CK(hipEventSynchronize(b));
  float ms = 0;
  CK(hipEventElapsedTime(&ms, a, b));
  CK(hipMemcpy(host_out, out, sizeof(host_out), hipMemcpyDeviceToHost));
  uint64_t sum = 0;
  for (uint32_t i = 0; i < lanes; ++i) sum += host_out[i];
  const double g = double(lanes) * steps / (ms * 1e-3);
  std::printf("| %-34s | %10.1f | %8.3f | %7.1f | %llu |\n", what, n * 16.0 / 1e6, ms, g / 1e9,
              (unsigned long long)sum);
  return 0;
}

template <int K>
int run_chains(const v4i *t, uint32_t n, uint32_t g, uint32_t lanes, uint32_t *out, hipEvent_t a, hipEvent_t b) {
  const int steps = 32;
  chase_chains<K><<<lanes / 256, 256>>>(t, n, g, steps, out);
  CK(hipDeviceSynchronize());
  CK(hipEventRecord(a));
  chase_chains<K><<<lanes / 256, 256>>>(t, n, g, steps, out);
  CK(hipEventRecord(b));
  CK(hipEventSynchronize(b));
  float ms = 0;
  CK(hipEventElapsedTime(&ms, a, b));
  CK(hipMemcpy(host_out, out, lanes * sizeof(uint32_t), hipMemcpyDeviceToHost));
  uint64_t sum = 0;
  for (uint32_t i = 0; i < lanes; ++i) sum += host_out[i];
  const double g_per_s = double(lanes) * steps * K / (ms * 1e-3);
  std::printf("| %10.1f | %6u | %10.1f | %9u | %6d | %8.3f | %7.1f | %llu |\n", n * 16.0 / 1e6, g,
              n * 16.0 * g / 1e6, lanes, K, ms, g_per_s / 1e9, (unsigned long long)sum);
  std::fflush(stdout);
  return 0;
}

int main() {
  hipDeviceProp_t prop;
  CK(hipGetDeviceProperties(&prop, 0));
  std::printf("device %s, %d CUs, %d MHz, L2 %d MB\n\n", prop.gcnArchName, prop.multiProcessorCount,
              prop.clockRate / 1000, prop.l2CacheSize >> 20);
  const uint64_t maxn = 1ull << 28;  // 4 GiB of 16-byte records
  v4i *t;
  CK(hipMalloc(&t, maxn * sizeof(v4i)));
  uint32_t *out;
  CK(hipMalloc(&out, sizeof(host_out)));
  hipEvent_t a, b;
  CK(hipEventCreate(&a));
  CK(hipEventCreate(&b));

  {  // streaming copy, 2 GiB read + 2 GiB written
    const uint64_t n = (1ull << 31) / sizeof(v4i);
    copy16<<<8192, 256>>>(t, t + n, n);
    CK(hipDeviceSynchronize());
    CK(hipEventRecord(a));
    for (int r = 0; r < 5; ++r) copy16<<<8192, 256>>>(t, t + n, n);
    CK(hipEventRecord(b));
    CK(hipEventSynchronize(b));
    float ms = 0;
    CK(hipEventElapsedTime(&ms, a, b));
    ms /= 5;
    std::printf("copy 2 GiB -> 2 GiB: %.3f ms, %.0f GB/s read+write\n\n", ms, 2.0 * (1ull << 31) / (ms * 1e6));
  }

  std::printf("2M lanes x 32 dependent reads each\n\n");
  std::printf("| %-34s | %10s | %8s | %7s | %s |\n", "read", "table MB", "ms", "G/s", "checksum");
  std::printf("|---|---|---|---|---|\n");
  const uint64_t sizes[] = {1ull << 15, 1ull << 18, 1ull << 20, 10000000ull, 1ull << 24, 1ull << 28};
  for (uint64_t n : sizes) {
    fill<<<4096, 256>>>(t, n);
    CK(hipDeviceSynchronize());
    if (run<0>(t, n, out, "8 B", a, b)) return 1;
    if (run<1>(t, n, out, "16 B", a, b)) return 1;
    if (n == 10000000ull) {
      if (run<2>(t, n, out, "8 B non-temporal", a, b)) return 1;
      if (run<3>(t, n, out, "8 B buffer sc0 sc1", a, b)) return 1;
    }
  }
  const uint64_t n = 10000000ull;  // 160 MB
  v4i *tf, *tu;
  CK(hipExtMallocWithFlags((void **)&tf, n * sizeof(v4i), hipDeviceMallocFinegrained));
  fill<<<4096, 256>>>(tf, n);
  CK(hipDeviceSynchronize());
  if (run<0>(tf, n, out, "8 B, fine-grained memory", a, b)) return 1;
  CK(hipExtMallocWithFlags((void **)&tu, n * sizeof(v4i), hipDeviceMallocUncached));
  fill<<<4096, 256>>>(tu, n);
  CK(hipDeviceSynchronize());
  if (run<0>(tu, n, out, "8 B, uncached memory", a, b)) return 1;

  std::printf("\n16-byte dependent reads: working set (lines MB), spread factor (span MB = lines MB x spread),\n"
              "lanes and independent chains per lane; 32 reads per chain\n\n");
  std::printf("| lines MB | spread | span MB | lanes | chains | ms | G reads/s | checksum |\n");
  std::printf("|---|---|---|---|---|---|---|---|\n");
  struct Case {
    uint32_t n, g;
  };
  const Case cases[] = {
      {1u << 18, 1},  {1u << 18, 16}, {1u << 18, 256}, {1u << 20, 1},  {1u << 20, 4},  {1u << 20, 16},
      {1u << 20, 64}, {1u << 20, 256}, {1u << 21, 1},  {1u << 21, 64}, {1u << 22, 1},  {1u << 22, 32},
      {6u << 20, 1},  {10u << 20, 1}, {1u << 24, 1},   {1u << 28, 1},
  };
  const uint32_t full = 1u << 21;
  for (const Case &c : cases) {
    if (uint64_t(c.n) * c.g > maxn) continue;  // every index stays inside the 4 GiB table
    fill_spread<<<4096, 256>>>(t, c.n, c.g);
    CK(hipDeviceSynchronize());
    if (run_chains<1>(t, c.n, c.g, full, out, a, b)) return 1;
    if (c.g == 1 && (c.n == (10u << 20) || c.n == (1u << 28))) {
      if (run_chains<2>(t, c.n, c.g, full, out, a, b)) return 1;
      if (run_chains<4>(t, c.n, c.g, full, out, a, b)) return 1;
      if (run_chains<1>(t, c.n, c.g, full / 4, out, a, b)) return 1;
      if (run_chains<1>(t, c.n, c.g, full / 8, out, a, b)) return 1;
      if (run_chains<1>(t, c.n, c.g, full / 16, out, a, b)) return 1;
      if (run_chains<4>(t, c.n, c.g, full / 16, out, a, b)) return 1;
    }
  }
  return 0;
}
