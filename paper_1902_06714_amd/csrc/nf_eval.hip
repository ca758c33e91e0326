// Classification count of section 4: a sample is correct when its output row
// and its target row have their largest entry at the same index.
#include <hip/hip_runtime.h>

#include "nf_internal.h"

namespace nf {
namespace {

constexpr int EVAL_WAVES = 4;

template <class T>
struct ArgMax {
  T v;
  int i;     // -1: empty
  bool nan;
};

// first index among equal largest entries; the order of combination does
// not matter because ties go to the smaller index
template <class T>
__device__ inline ArgMax<T> better(ArgMax<T> a, ArgMax<T> b) {
  ArgMax<T> r;
  r.nan = a.nan || b.nan;
  const bool take_b = b.i >= 0 && (a.i < 0 || b.v > a.v || (b.v == a.v && b.i < a.i));
  r.v = take_b ? b.v : a.v;
  r.i = take_b ? b.i : a.i;
  return r;
}

template <class T>
__device__ inline ArgMax<T> wave_argmax(const T* row, int n, int lane) {
  ArgMax<T> m{T(0), -1, false};
  for (int j = lane; j < n; j += 64) {
    const T v = row[j];
    if (v != v) m.nan = true;
    else m = better(m, ArgMax<T>{v, j, false});
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    ArgMax<T> o;
    o.v = __shfl_xor(m.v, off, 64);
    o.i = __shfl_xor(m.i, off, 64);
    o.nan = __shfl_xor((int)m.nan, off, 64) != 0;
    m = better(m, o);
  }
  return m;
}

// One wave per sample row; every workgroup adds its count once.
template <class T>
__global__ __launch_bounds__(64 * EVAL_WAVES) void count_correct_kernel(
    const T* __restrict__ out, int64_t ldo, const T* __restrict__ y, int64_t ldy, int64_t n,
    int d, unsigned long long* __restrict__ count) {
  __shared__ int wave_hits[EVAL_WAVES];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int hits = 0;
  for (int64_t s = (int64_t)blockIdx.x * EVAL_WAVES + wave; s < n;
       s += (int64_t)gridDim.x * EVAL_WAVES) {
    const ArgMax<T> a = wave_argmax(out + s * ldo, d, lane);
    const ArgMax<T> t = wave_argmax(y + s * ldy, d, lane);
    hits += (!a.nan && !t.nan && a.i >= 0 && a.i == t.i) ? 1 : 0;
  }
  if (lane == 0) wave_hits[wave] = hits;
  __syncthreads();
  if (threadIdx.x == 0) {
    int sum = 0;
#pragma unroll
    for (int w = 0; w < EVAL_WAVES; ++w) sum += wave_hits[w];
    if (sum) atomicAdd(count, (unsigned long long)sum);
  }
}

}  // namespace

template <class T>
hipError_t launch_count_correct(const T* out, int64_t ldo, const T* y, int64_t ldy, int64_t n,
                                int d, unsigned long long* count, hipStream_t s) {
  if (n <= 0 || d <= 0) return hipErrorInvalidValue;
  const int64_t want = (n + EVAL_WAVES - 1) / EVAL_WAVES;
  const int blocks = (int)(want < 2048 ? want : 2048);
  return launch_k(count_correct_kernel<T>, blocks, 64 * EVAL_WAVES, 0, s, out, ldo, y, ldy, n, d,
                  count);
}

template hipError_t launch_count_correct<float>(const float*, int64_t, const float*, int64_t,
                                                int64_t, int, unsigned long long*, hipStream_t);
template hipError_t launch_count_correct<double>(const double*, int64_t, const double*, int64_t,
                                                 int64_t, int, unsigned long long*, hipStream_t);

}  // namespace nf
