// Measurement aids: the device peaks that the roofline fractions are measured
// against (include/nf.h, nf_calib_*).  A streaming read, a streaming copy and
// a loop of independent matrix-core instructions, each timed by the kernel's
// own start and end.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "nf.h"
#include "nf_internal.h"

namespace nf {

constexpr int CAL_THREADS = 256;
constexpr int CAL_UNROLL = 4;

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef double doublex4 __attribute__((ext_vector_type(4)));

// every thread reads 16-byte vectors CAL_UNROLL at a time, grid-strided;
// one float per workgroup keeps the loads live
__global__ void __launch_bounds__(CAL_THREADS) calib_read_kernel(const float4* src, int64_t n16,
                                                                  float* sink) {
  const int64_t stride = (int64_t)gridDim.x * CAL_THREADS;
  int64_t i = (int64_t)blockIdx.x * CAL_THREADS + threadIdx.x;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (; i + (CAL_UNROLL - 1) * stride < n16; i += CAL_UNROLL * stride) {
    float4 v[CAL_UNROLL];
#pragma unroll
    for (int u = 0; u < CAL_UNROLL; ++u) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < CAL_UNROLL; ++u) {
      acc.x += v[u].x;
      acc.y += v[u].y;
      acc.z += v[u].z;
      acc.w += v[u].w;
    }
  }
  for (; i < n16; i += stride) {
    const float4 v = src[i];
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  __shared__ float red[CAL_THREADS];
  red[threadIdx.x] = (acc.x + acc.y) + (acc.z + acc.w);
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.0f;
    for (int k = 0; k < CAL_THREADS; ++k) t += red[k];
    sink[blockIdx.x] = t;
  }
}

__global__ void __launch_bounds__(CAL_THREADS) calib_copy_kernel(float4* dst, const float4* src,
                                                                  int64_t n16) {
  const int64_t stride = (int64_t)gridDim.x * CAL_THREADS;
  int64_t i = (int64_t)blockIdx.x * CAL_THREADS + threadIdx.x;
  for (; i + (CAL_UNROLL - 1) * stride < n16; i += CAL_UNROLL * stride) {
    float4 v[CAL_UNROLL];
#pragma unroll
    for (int u = 0; u < CAL_UNROLL; ++u) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < CAL_UNROLL; ++u) dst[i + u * stride] = v[u];
  }
  for (; i < n16; i += stride) dst[i] = src[i];
}

// CAL_CHAINS independent accumulators per wave, each a chain of `iters`
// matrix instructions; wave 0 of each workgroup stamps the shader clock
// (s_memtime) and the 100 MHz constant clock (s_memrealtime) at its start and
// end, so the host can tell the clock the matrix cores ran at
constexpr int CAL_CHAINS = 8;
constexpr int CAL_GROUP = 8;     // rounds per loop trip; iters is rounded up to a multiple
// workgroups of 4 waves per CU: two waves per SIMD for fp32 (128 accumulator
// registers each), four for fp64 (64 each), whose chains need more in flight
constexpr int CAL_MFMA_WG32 = 2, CAL_MFMA_WG64 = 4;

template <bool F64>
__global__ void __launch_bounds__(CAL_THREADS) calib_mfma_kernel(int64_t iters, float* sink,
                                                                  uint64_t* stamps) {
  const int lane = threadIdx.x & 63;
  uint64_t c0 = 0, r0 = 0;
  if (threadIdx.x == 0) {
    c0 = __builtin_amdgcn_s_memtime();
    r0 = __builtin_amdgcn_s_memrealtime();
  }
  float total = 0.0f;
  if constexpr (!F64) {
    const float a = 1.0f + 1e-7f * lane, b = 1.0f - 1e-7f * lane;
    floatx16 acc[CAL_CHAINS];
#pragma unroll
    for (int c = 0; c < CAL_CHAINS; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[c][v] = 0.0f;
    // whole groups of CAL_GROUP rounds per trip: the compiler moves the
    // accumulators between register files at the loop's back edge
    for (int64_t it = 0; it < iters; it += CAL_GROUP)
#pragma unroll
      for (int r = 0; r < CAL_GROUP; ++r)
#pragma unroll
        for (int c = 0; c < CAL_CHAINS; ++c)
          acc[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[c], 0, 0, 0);
#pragma unroll
    for (int c = 0; c < CAL_CHAINS; ++c) total += acc[c][lane & 15];
  } else {
    const double a = 1.0 + 1e-9 * lane, b = 1.0 - 1e-9 * lane;
    doublex4 acc[CAL_CHAINS];
#pragma unroll
    for (int c = 0; c < CAL_CHAINS; ++c)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[c][v] = 0.0;
    for (int64_t it = 0; it < iters; it += CAL_GROUP)
#pragma unroll
      for (int r = 0; r < CAL_GROUP; ++r)
#pragma unroll
        for (int c = 0; c < CAL_CHAINS; ++c)
          acc[c] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc[c], 0, 0, 0);
#pragma unroll
    for (int c = 0; c < CAL_CHAINS; ++c) total += (float)acc[c][lane & 3];
  }
  if (lane == 0) sink[(int64_t)blockIdx.x * (CAL_THREADS / 64) + (threadIdx.x >> 6)] = total;
  if (threadIdx.x == 0) {
    const uint64_t c1 = __builtin_amdgcn_s_memtime();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
    uint64_t* st = stamps + 4 * (int64_t)blockIdx.x;
    st[0] = c0;
    st[1] = c1;
    st[2] = r0;
    st[3] = r1;
  }
}

// One wave that returns once `ticks` of the 100 MHz constant clock have
// passed since it started (bounded by the caller to one second).
__global__ void __launch_bounds__(64) calib_spin_kernel(uint64_t ticks) {
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  while (__builtin_amdgcn_s_memrealtime() - t0 < ticks) __builtin_amdgcn_s_sleep(8);
}

}  // namespace nf

namespace {

nf_status cfail(nf_status st, const std::string& m) {
  nf::set_error_message(m.c_str());
  return st;
}

int device_cus() {
  int dev = 0, ncu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  return ncu;
}

// runs enqueue() with a pair of events bound to its kernel, waits, returns ms
template <class F>
nf_status time_one(hipStream_t s, double* host_ms, F&& enqueue) {
  hipEvent_t a = nullptr, b = nullptr;
  hipError_t e = hipEventCreate(&a);
  if (e == hipSuccess) e = hipEventCreate(&b);
  if (e == hipSuccess) {
    nf::launch_events() = {a, b};
    e = enqueue();
    nf::launch_events() = {};
  }
  if (e == hipSuccess) e = hipEventSynchronize(b);
  float ms = 0.0f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return cfail(NF_EDEVICE, std::string("calibration kernel: ") + hipGetErrorString(e));
  }
  *host_ms = ms;
  return NF_OK;
}

}  // namespace

extern "C" {

nf_status nf_calib_read(const void* d_src, int64_t bytes, void* d_sink, void* stream,
                        double* host_ms) {
  nf::set_error_message("");
  if (!d_src || !d_sink || !host_ms) return cfail(NF_EINVAL, "NULL pointer");
  if (bytes <= 0 || bytes % 16 != 0 || (reinterpret_cast<uintptr_t>(d_src) & 15) != 0)
    return cfail(NF_EINVAL, "bytes must be a positive multiple of 16 at a 16-byte address");
  const int ncu = device_cus();
  if (ncu <= 0) return cfail(NF_EDEVICE, "no usable HIP device");
  const int grid = 4 * ncu;
  if ((int64_t)grid * 4 > NF_CALIB_SINK_BYTES) return cfail(NF_ESHAPE, "sink too small");
  return time_one(static_cast<hipStream_t>(stream), host_ms, [&] {
    return nf::launch_k(nf::calib_read_kernel, dim3(grid), dim3(nf::CAL_THREADS), 0,
                        static_cast<hipStream_t>(stream), static_cast<const float4*>(d_src),
                        bytes / 16, static_cast<float*>(d_sink));
  });
}

nf_status nf_calib_copy(void* d_dst, const void* d_src, int64_t bytes, void* stream,
                        double* host_ms) {
  nf::set_error_message("");
  if (!d_src || !d_dst || !host_ms) return cfail(NF_EINVAL, "NULL pointer");
  if (bytes <= 0 || bytes % 16 != 0 || ((reinterpret_cast<uintptr_t>(d_src) |
                                         reinterpret_cast<uintptr_t>(d_dst)) & 15) != 0)
    return cfail(NF_EINVAL, "bytes must be a positive multiple of 16 at 16-byte addresses");
  const int ncu = device_cus();
  if (ncu <= 0) return cfail(NF_EDEVICE, "no usable HIP device");
  return time_one(static_cast<hipStream_t>(stream), host_ms, [&] {
    return nf::launch_k(nf::calib_copy_kernel, dim3(4 * ncu), dim3(nf::CAL_THREADS), 0,
                        static_cast<hipStream_t>(stream), static_cast<float4*>(d_dst),
                        static_cast<const float4*>(d_src), bytes / 16);
  });
}

nf_status nf_calib_mfma(int32_t dtype, int64_t iters, void* d_sink, void* stream,
                        double* host_ms, double* host_flops, double* host_clock_ghz) {
  nf::set_error_message("");
  if (!d_sink || !host_ms || !host_flops || !host_clock_ghz)
    return cfail(NF_EINVAL, "NULL pointer");
  if (dtype != NF_F32 && dtype != NF_F64) return cfail(NF_EINVAL, "unknown dtype");
  if (iters < 1 || iters > ((int64_t)1 << 30)) return cfail(NF_EINVAL, "iters out of range");
  iters = (iters + nf::CAL_GROUP - 1) / nf::CAL_GROUP * nf::CAL_GROUP;
  const int ncu = device_cus();
  if (ncu <= 0) return cfail(NF_EDEVICE, "no usable HIP device");
  const int grid = (dtype == NF_F64 ? nf::CAL_MFMA_WG64 : nf::CAL_MFMA_WG32) * ncu;
  const int64_t sink_floats = (int64_t)grid * (nf::CAL_THREADS / 64);
  const int64_t need = sink_floats * 4 + (int64_t)grid * 32;
  if (need > NF_CALIB_SINK_BYTES) return cfail(NF_ESHAPE, "sink too small for this device");
  float* sink = static_cast<float*>(d_sink);
  uint64_t* stamps = reinterpret_cast<uint64_t*>(sink + sink_floats);
  hipStream_t s = static_cast<hipStream_t>(stream);
  nf_status st = time_one(s, host_ms, [&] {
    return dtype == NF_F64
               ? nf::launch_k(nf::calib_mfma_kernel<true>, dim3(grid), dim3(nf::CAL_THREADS), 0,
                              s, iters, sink, stamps)
               : nf::launch_k(nf::calib_mfma_kernel<false>, dim3(grid), dim3(nf::CAL_THREADS), 0,
                              s, iters, sink, stamps);
  });
  if (st != NF_OK) return st;
  // 4 waves per workgroup, CAL_CHAINS instructions per iteration; 2 flops per
  // multiply-add of a 32x32x2 (fp32) or 16x16x4 (fp64) block
  const double per = dtype == NF_F64 ? 2.0 * 16 * 16 * 4 : 2.0 * 32 * 32 * 2;
  *host_flops = (double)grid * 4 * nf::CAL_CHAINS * (double)iters * per;
  std::vector<uint64_t> h(4 * (size_t)grid);
  const int nread = grid;
  hipError_t e = hipMemcpy(h.data(), stamps, (size_t)nread * 32, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return cfail(NF_EDEVICE, std::string("stamps: ") + hipGetErrorString(e));
  double sum = 0.0;
  int used = 0;
  for (int i = 0; i < nread; ++i) {
    const double dc = (double)(h[4 * i + 1] - h[4 * i]), dr = (double)(h[4 * i + 3] - h[4 * i + 2]);
    if (dr > 0) {
      sum += dc / dr * 0.1;   // constant clock at 100 MHz: GHz = cycles per tick / 10
      ++used;
    }
  }
  *host_clock_ghz = used ? sum / used : 0.0;
  return NF_OK;
}

nf_status nf_calib_spin(void* stream, double us) {
  nf::set_error_message("");
  if (!(us >= 0.0 && us <= 1e6)) return cfail(NF_EINVAL, "us must be in 0 .. 1e6");
  const hipError_t e = nf::launch_k(nf::calib_spin_kernel, dim3(1), dim3(64), 0,
                                    static_cast<hipStream_t>(stream), (uint64_t)(us * 100.0));
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return cfail(NF_EDEVICE, std::string("spin kernel: ") + hipGetErrorString(e));
  }
  return NF_OK;
}

}  // extern "C"
