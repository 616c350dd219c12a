// Device probes behind kf_probe_bandwidth / kf_probe_overhead (paper Section
// V-A: the bandwidth and the per-token dispatch overhead of eq. (2) are
// measured on the device before any weight is loaded).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <vector>

#include "error.h"
#include "kafila_planner.h"

using kf::fail;

namespace {

typedef unsigned v4u __attribute__((ext_vector_type(4)));

constexpr int kProbeThreads = 256;
constexpr int64_t kProbeSpan = 64 * 1024;  // bytes per workgroup per pass

// Streams the buffer with 16-byte non-temporal loads, the access the decode
// GEMVs make: workgroup w reads spans w, w + grid, ...; each thread 16 B of every
// 4 KB stride of its span.  The xor of everything read goes to out[w] so that no
// load is dead.
__global__ __launch_bounds__(kProbeThreads) void hbm_read_probe_kernel(const v4u* __restrict__ buf, int64_t spans,
                                                                       unsigned* __restrict__ out) {
  constexpr int per_span = (int)(kProbeSpan / 16);  // 16-byte chunks per span
  unsigned acc = 0;
  for (int64_t s = blockIdx.x; s < spans; s += gridDim.x) {
    const v4u* p = buf + s * per_span;
#pragma unroll 4
    for (int c = threadIdx.x; c < per_span; c += kProbeThreads) {
      const v4u v = __builtin_nontemporal_load(p + c);
      acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
  }
  __shared__ unsigned red[kProbeThreads];
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned a = 0;
    for (int i = 0; i < kProbeThreads; ++i) a ^= red[i];
    out[blockIdx.x] = a;
  }
}

__global__ void empty_kernel() {}

double median(std::vector<double> v) {
  std::sort(v.begin(), v.end());
  const size_t n = v.size();
  return n % 2 ? v[n / 2] : 0.5 * (v[n / 2 - 1] + v[n / 2]);
}

struct Events {
  hipEvent_t a = nullptr, b = nullptr;
  ~Events() {
    if (a) (void)hipEventDestroy(a);
    if (b) (void)hipEventDestroy(b);
  }
};

}  // namespace

#define KF_PROBE_HIP(call, what)                                                            \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess) return fail(KF_EDEVICE, "%s: %s", (what), hipGetErrorString(e_)); \
  } while (0)

extern "C" {

kf_status kf_probe_bandwidth(void* hip_stream, int64_t bytes, int32_t reps, double* bw) {
  if (!bw) return fail(KF_EINVAL, "bw is NULL");
  if (reps < 1) return fail(KF_EINVAL, "reps must be >= 1");
  if (bytes < (64LL << 20) || bytes % kProbeSpan) return fail(KF_EINVAL, "bytes must be >= 64 MiB and a multiple of 64 KiB");
  hipStream_t st = (hipStream_t)hip_stream;
  const int64_t spans = bytes / kProbeSpan;
  int dev = 0, cus = 0;
  KF_PROBE_HIP(hipGetDevice(&dev), "hipGetDevice");
  KF_PROBE_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev), "hipDeviceGetAttribute");
  // Eight workgroups per CU, never more than there are spans.
  const int grid = (int)std::min<int64_t>(spans, std::max(2048, 8 * cus));

  void* buf = nullptr;
  unsigned* out = nullptr;
  if (hipMalloc(&buf, (size_t)bytes) != hipSuccess) {
    (void)hipGetLastError();
    return fail(KF_ENOMEM, "probe buffer of %lld bytes", (long long)bytes);
  }
  if (hipMalloc((void**)&out, (size_t)grid * sizeof(unsigned)) != hipSuccess) {
    (void)hipGetLastError();
    (void)hipFree(buf);
    return fail(KF_ENOMEM, "probe output");
  }
  kf_status result = KF_OK;
  {
    Events ev;
    std::vector<double> t;
    hipError_t e = hipMemsetAsync(buf, 0x5a, (size_t)bytes, st);
    if (e == hipSuccess) e = hipEventCreate(&ev.a);
    if (e == hipSuccess) e = hipEventCreate(&ev.b);
    for (int r = 0; r <= reps && e == hipSuccess; ++r) {
      e = hipEventRecord(ev.a, st);
      if (e == hipSuccess) {
        hipLaunchKernelGGL(hbm_read_probe_kernel, dim3(grid), dim3(kProbeThreads), 0, st, (const v4u*)buf, spans, out);
        e = hipGetLastError();
      }
      if (e == hipSuccess) e = hipEventRecord(ev.b, st);
      if (e == hipSuccess) e = hipEventSynchronize(ev.b);
      float ms = 0;
      if (e == hipSuccess) e = hipEventElapsedTime(&ms, ev.a, ev.b);
      if (e == hipSuccess && r > 0) t.push_back(ms * 1e-3);
    }
    if (e != hipSuccess) result = fail(KF_EDEVICE, "bandwidth probe: %s", hipGetErrorString(e));
    else *bw = (double)bytes / median(t);
  }
  (void)hipFree(out);
  (void)hipFree(buf);
  return result;
}

kf_status kf_probe_overhead(void* hip_stream, int32_t reps, double* o) {
  if (!o) return fail(KF_EINVAL, "o is NULL");
  if (reps < 1) return fail(KF_EINVAL, "reps must be >= 1");
  constexpr int kChain = 256;
  hipStream_t st = (hipStream_t)hip_stream;
  Events ev;
  KF_PROBE_HIP(hipEventCreate(&ev.a), "hipEventCreate");
  KF_PROBE_HIP(hipEventCreate(&ev.b), "hipEventCreate");
  std::vector<double> t;
  for (int r = 0; r <= reps; ++r) {
    KF_PROBE_HIP(hipEventRecord(ev.a, st), "hipEventRecord");
    for (int i = 0; i < kChain; ++i) hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, st);
    KF_PROBE_HIP(hipGetLastError(), "empty kernel launch");
    KF_PROBE_HIP(hipEventRecord(ev.b, st), "hipEventRecord");
    KF_PROBE_HIP(hipEventSynchronize(ev.b), "hipEventSynchronize");
    float ms = 0;
    KF_PROBE_HIP(hipEventElapsedTime(&ms, ev.a, ev.b), "hipEventElapsedTime");
    if (r > 0) t.push_back(ms * 1e-3 / kChain);
  }
  *o = median(t);
  return KF_OK;
}

}  // extern "C"
