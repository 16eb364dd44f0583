// Streaming ceilings for the benchmark (libacp_probe.so, not part of the compressor): the access
// mix of the compress kernels (read M, read E, write E in place, every access nontemporal) and of
// the decompress kernels (write only, nontemporal), over arrays much larger than the caches.
// A workgroup moves 4, 8, 16 or 32 KB of each stream (the footprints the kernels' tiles walk
// with), chosen per call; the grid covers the arrays once.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr int kThreads = 256;
typedef float v4f __attribute__((ext_vector_type(4)));

// kPerThread 16-byte vectors per thread and stream: kPerThread * 4 KB per workgroup
template <int kPerThread>
__global__ __launch_bounds__(kThreads) void k_probe_rrw(const v4f* __restrict__ m, v4f* __restrict__ e,
                                                        int64_t n4) {
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kPerThread * kThreads + threadIdx.x;
  v4f a[kPerThread], b[kPerThread];
#pragma unroll
  for (int u = 0; u < kPerThread; ++u) {
    const int64_t i = base + static_cast<int64_t>(u) * kThreads;
    if (i < n4) {
      a[u] = __builtin_nontemporal_load(m + i);
      b[u] = __builtin_nontemporal_load(e + i);
    }
  }
#pragma unroll
  for (int u = 0; u < kPerThread; ++u) {
    const int64_t i = base + static_cast<int64_t>(u) * kThreads;
    if (i < n4) {
      __builtin_nontemporal_store(a[u] + b[u], e + i);
    }
  }
}

template <int kPerThread>
__global__ __launch_bounds__(kThreads) void k_probe_w(v4f* __restrict__ out, int64_t n4, float v) {
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kPerThread * kThreads + threadIdx.x;
  const v4f s = {v, v, v, v};
#pragma unroll
  for (int u = 0; u < kPerThread; ++u) {
    const int64_t i = base + static_cast<int64_t>(u) * kThreads;
    if (i < n4) __builtin_nontemporal_store(s, out + i);
  }
}

dim3 grid_of(int64_t n4, int per_thread) {
  return dim3(static_cast<unsigned>((n4 + per_thread * kThreads - 1) / (per_thread * kThreads)));
}

template <typename K1, typename K2, typename K4, typename K8>
bool pick(int kb, K1 k1, K2 k2, K4 k4, K8 k8) {
  switch (kb) {
    case 4: k1(); return true;
    case 8: k2(); return true;
    case 16: k4(); return true;
    case 32: k8(); return true;
    default: return false;
  }
}

}  // namespace

extern "C" {

// e[i] = m[i] + e[i] for i < n (n a multiple of 4, both 16-byte aligned device arrays), each
// workgroup taking kb KB of each array (kb = 4, 8, 16 or 32); returns a hipError_t.
int acp_probe_rrw(const float* m, float* e, int64_t n, int kb, void* stream) {
  if (!m || !e || n <= 0 || (n & 3)) return static_cast<int>(hipErrorInvalidValue);
  const int64_t n4 = n / 4;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const v4f* mv = reinterpret_cast<const v4f*>(m);
  v4f* ev = reinterpret_cast<v4f*>(e);
  const bool ok = pick(
      kb, [&] { hipLaunchKernelGGL(k_probe_rrw<1>, grid_of(n4, 1), dim3(kThreads), 0, s, mv, ev, n4); },
      [&] { hipLaunchKernelGGL(k_probe_rrw<2>, grid_of(n4, 2), dim3(kThreads), 0, s, mv, ev, n4); },
      [&] { hipLaunchKernelGGL(k_probe_rrw<4>, grid_of(n4, 4), dim3(kThreads), 0, s, mv, ev, n4); },
      [&] { hipLaunchKernelGGL(k_probe_rrw<8>, grid_of(n4, 8), dim3(kThreads), 0, s, mv, ev, n4); });
  if (!ok) return static_cast<int>(hipErrorInvalidValue);
  return static_cast<int>(hipGetLastError());
}

// out[i] = v for i < n (n a multiple of 4, 16-byte aligned device array), each workgroup writing
// kb KB (kb = 4, 8, 16 or 32); returns a hipError_t.
int acp_probe_w(float* out, int64_t n, float v, int kb, void* stream) {
  if (!out || n <= 0 || (n & 3)) return static_cast<int>(hipErrorInvalidValue);
  const int64_t n4 = n / 4;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  v4f* ov = reinterpret_cast<v4f*>(out);
  const bool ok = pick(
      kb, [&] { hipLaunchKernelGGL(k_probe_w<1>, grid_of(n4, 1), dim3(kThreads), 0, s, ov, n4, v); },
      [&] { hipLaunchKernelGGL(k_probe_w<2>, grid_of(n4, 2), dim3(kThreads), 0, s, ov, n4, v); },
      [&] { hipLaunchKernelGGL(k_probe_w<4>, grid_of(n4, 4), dim3(kThreads), 0, s, ov, n4, v); },
      [&] { hipLaunchKernelGGL(k_probe_w<8>, grid_of(n4, 8), dim3(kThreads), 0, s, ov, n4, v); });
  if (!ok) return static_cast<int>(hipErrorInvalidValue);
  return static_cast<int>(hipGetLastError());
}

}  // extern "C"
