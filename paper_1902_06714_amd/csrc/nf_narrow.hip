// Training step for narrow networks (every layer after the input has at most
// 32 units, like the paper's 784-30-10 MNIST network, section 4).
//
// Kernel 1, per 16-sample tile (one workgroup of 8 waves):
//   layer 1   z_1 = W_1 x + b_1 on the fp32 matrix cores (16x16x4), the input
//             width staged through LDS in 128-wide chunks, each wave taking one
//             16-wide group per chunk, the waves' sums added in wave order;
//   layers 2+ one thread per (sample, unit) with the previous layer in LDS;
//   deltas    output delta (a_L - y) f'(z_L) and hidden deltas
//             (W_{l+1}^T delta_{l+1}) f'(z_l) (section 3.3), with f'(z_l) kept
//             in registers from the forward pass.
// Kernel 2, tendencies of every layer (sections 3.3-3.5): workgroup
//   (layer, 16-column tile, 16-unit half) forms the batch sum of delta (outer)
//   activation for its block on the matrix cores (16x16x4), its 8 waves
//   splitting the batch and their sums added in wave order; it then stores the tendency and
//   writes W' = W - (eta/B) G itself (into the other parameter buffer), so no
//   workgroup waits on another.  The order of every sum is fixed, so results
//   are reproducible bit for bit.
#include "nf_act.h"
#include "nf_internal.h"

namespace nf {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

// v if c, else zeros; written per component (a conditional on the vector
// type itself is lowered through private memory)
__device__ __forceinline__ float4 keep_if(bool c, float4 v) {
  return make_float4(c ? v.x : 0.0f, c ? v.y : 0.0f, c ? v.z : 0.0f, c ? v.w : 0.0f);
}

constexpr int N1_WAVES = 8;
constexpr int N1_KC = 16 * N1_WAVES;  // inputs per LDS stage: one 16-wide group per wave
constexpr int N1_KP = N1_KC + 4;      // padded LDS row
// chunks requested together: 8 for training (one launch of few workgroups),
// 4 for inference (fewer registers, two workgroups per CU)
constexpr int N1_PRE_TRAIN = 8;
constexpr int N1_PRE_INFER = 4;

template <bool TRAIN, int N1_PRE>
__global__ void __launch_bounds__(N1_WAVES * 64) narrow_fwd_kernel(const NarrowFwdParams p) {
  constexpr int T = NARROW_TILE;
  constexpr int NW = NARROW_WIDTH;
  // layer-1 staging (input chunk xs, W_1 chunk wsl, two buffers each); the
  // per-wave partial sums zp reuse the same bytes once layer 1 is done
  __shared__ __attribute__((aligned(16))) float stage[2 * (T + NW) * N1_KP];
  static_assert(N1_WAVES * T * (NW + 1) <= 2 * (T + NW) * N1_KP, "zp must fit the staging area");
  auto xs = reinterpret_cast<float(*)[T][N1_KP]>(stage);
  auto wsl = reinterpret_cast<float(*)[NW][N1_KP]>(stage + 2 * T * N1_KP);
  auto zp = reinterpret_cast<float(*)[T][NW + 1]>(stage);
  __shared__ float hs[2][T][NW + 1];                         // activations, then deltas
  __shared__ float ws[NARROW_MAX_LAYERS - 1][NW][NW + 1];    // W_2 .. W_L
  __shared__ float bs[NARROW_MAX_LAYERS][NW];                // b_1 .. b_L

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int s0 = blockIdx.x * T;

  // stage the small layers' weights and every bias in LDS (read again and
  // again by the per-sample threads below).  The layer loops are unrolled so
  // that every kernel-argument index is a constant; the loads are issued
  // together and land while layer 1 runs.  Out-of-range entries read W_1[0][0]
  // (always present) and are zeroed.
  constexpr int NPER = NW * NW / (N1_WAVES * 64);
  static_assert(NW * NW % (N1_WAVES * 64) == 0, "staging split");
  float wst[NARROW_MAX_LAYERS - 1][NPER];
#pragma unroll
  for (int li = 0; li < NARROW_MAX_LAYERS - 1; ++li) {
    const int l = li + 2;
#pragma unroll
    for (int u = 0; u < NPER; ++u) {
      const int e = tid + u * N1_WAVES * 64, row = e / NW, colw = e % NW;
      const bool ok = l <= p.L && row < p.dims[l] && colw < p.dims[l - 1];
      const float* src = ok ? p.W[l - 1] + (int64_t)row * p.ldw[l - 1] + colw : p.W[0];
      const float v = *src;
      wst[li][u] = ok ? v : 0.0f;
    }
  }
  float bst[NARROW_MAX_LAYERS];
#pragma unroll
  for (int l = 1; l <= NARROW_MAX_LAYERS; ++l) {
    const int u = tid & (NW - 1);
    const bool ok = l <= p.L && u < p.dims[l];
    const float* src = ok ? p.bias[l - 1] + u : p.W[0];
    const float v = *src;
    bst[l - 1] = ok ? v : 0.0f;
  }
  // this thread's target (sample tid / 32, output unit tid % 32)
  float ytg = 0.0f;
  if (TRAIN) {
    const int ys = s0 + (tid >> 5), yu = tid & 31;
    if (ys < p.B && yu < p.dims[p.L]) ytg = p.Y[(int64_t)ys * p.dims[p.L] + yu];
  }

  // ---- layer 1 on the matrix cores.  The inputs go through LDS in chunks of
  // N1_KC, read from global memory with contiguous full-line loads (X rows and
  // W_1 rows) that are all issued before the first chunk is used, and passed
  // through two LDS buffers chunk by chunk as the data arrives.
  // Wave w takes the w-th 16-wide group of every chunk; lane (r, g) =
  // (lane % 16, lane / 16) feeds sample r and units r, 16 + r with inputs
  // 4 g .. 4 g + 3 of the group, one per MFMA, so every product of the dot
  // product is formed.  Out-of-range rows and inputs are read from a valid
  // address and stored as zero.
  {
    const int r = lane & 15, g = lane >> 4;
    const int d1 = p.dims[1];
    const int nch = (p.d0 + N1_KC - 1) / N1_KC;
    // this thread's share of a chunk: one float4 of X, two of W_1
    const int xrow = tid / (N1_KC / 4), xq = tid % (N1_KC / 4);
    const bool xrow_ok = s0 + xrow < p.B;
    const float* xsrc = p.X + (int64_t)(xrow_ok ? s0 + xrow : p.B - 1) * p.d0;
    const bool w0_ok = xrow < d1, w1_ok = 16 + xrow < d1;
    const float* wsrc0 = p.W[0] + (int64_t)(w0_ok ? xrow : 0) * p.ldw[0];
    const float* wsrc1 = p.W[0] + (int64_t)(w1_ok ? 16 + xrow : 0) * p.ldw[0];
    // two accumulator chains per unit block (inputs 4g, 4g+2 and 4g+1, 4g+3
    // of each group) keep more MFMAs in flight; they are added at the end
    floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    floatx4 acc2 = {0.f, 0.f, 0.f, 0.f}, acc3 = {0.f, 0.f, 0.f, 0.f};
    // every chunk of a block of N1_PRE chunks is requested at once (one memory
    // latency per block); chunks then pass through LDS as they arrive
    for (int cb = 0; cb < nch; cb += N1_PRE) {
      float4 xr[N1_PRE], wr0[N1_PRE], wr1[N1_PRE];
#pragma unroll
      for (int u = 0; u < N1_PRE; ++u) {
        const int k = (cb + u) * N1_KC + 4 * xq;
        const bool k_ok = k < p.d0;
        const int kc = k_ok ? k : 0;
        const float4 xv = *reinterpret_cast<const float4*>(xsrc + kc);
        const float4 w0 = *reinterpret_cast<const float4*>(wsrc0 + kc);
        const float4 w1 = *reinterpret_cast<const float4*>(wsrc1 + kc);
        xr[u] = keep_if(k_ok && xrow_ok, xv);
        wr0[u] = keep_if(k_ok && w0_ok, w0);
        wr1[u] = keep_if(k_ok && w1_ok, w1);
      }
      // chunks past the input width were loaded as zeros, so the whole block
      // is processed unconditionally (keeps the loop fully unrolled)
#pragma unroll
      for (int u = 0; u < N1_PRE; ++u) {
        const int buf = u & 1;
        *reinterpret_cast<float4*>(&xs[buf][xrow][4 * xq]) = xr[u];
        *reinterpret_cast<float4*>(&wsl[buf][xrow][4 * xq]) = wr0[u];
        *reinterpret_cast<float4*>(&wsl[buf][16 + xrow][4 * xq]) = wr1[u];
        __syncthreads();
        const int ko = 16 * wave + 4 * g;
        const float4 x = *reinterpret_cast<const float4*>(&xs[buf][r][ko]);
        const float4 a = *reinterpret_cast<const float4*>(&wsl[buf][r][ko]);
        const float4 b = *reinterpret_cast<const float4*>(&wsl[buf][16 + r][ko]);
        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(x.x, a.x, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(x.x, b.x, acc1, 0, 0, 0);
        acc2 = __builtin_amdgcn_mfma_f32_16x16x4f32(x.y, a.y, acc2, 0, 0, 0);
        acc3 = __builtin_amdgcn_mfma_f32_16x16x4f32(x.y, b.y, acc3, 0, 0, 0);
        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(x.z, a.z, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(x.z, b.z, acc1, 0, 0, 0);
        acc2 = __builtin_amdgcn_mfma_f32_16x16x4f32(x.w, a.w, acc2, 0, 0, 0);
        acc3 = __builtin_amdgcn_mfma_f32_16x16x4f32(x.w, b.w, acc3, 0, 0, 0);
      }
      __syncthreads();   // the next block's first chunk reuses buffer 0
    }
    acc0 += acc2;
    acc1 += acc3;
    // accumulator register v of lane (r, g): sample 4 g + v, unit r (+16)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      zp[wave][4 * g + v][r] = acc0[v];
      zp[wave][4 * g + v][16 + r] = acc1[v];
    }
  }
#pragma unroll
  for (int li = 0; li < NARROW_MAX_LAYERS - 1; ++li)
#pragma unroll
    for (int u = 0; u < NPER; ++u) {
      const int e = tid + u * N1_WAVES * 64;
      ws[li][e / NW][e % NW] = wst[li][u];
    }
  if (tid < NW) {
#pragma unroll
    for (int l = 0; l < NARROW_MAX_LAYERS; ++l) bs[l][tid] = bst[l];
  }
  __syncthreads();

  // ---- thread (s, j): sample s of the tile, unit j of the current layer
  const int s = tid >> 5, j = tid & 31;
  const int gs = s0 + s;
  const bool s_ok = gs < p.B;
  float fp[NARROW_MAX_LAYERS];
#pragma unroll
  for (int l = 0; l < NARROW_MAX_LAYERS; ++l) fp[l] = 0.0f;
  int cur = 0;
  {
    float z = zp[0][s][j];
#pragma unroll
    for (int w = 1; w < N1_WAVES; ++w) z += zp[w][s][j];
    float a = 0.0f, f = 0.0f;
    if (j < p.dims[1]) act_eval(p.acts[0], z + bs[0][j], a, f);
    fp[0] = f;
    if (p.L == 1) {
      if (TRAIN) {
        const float d = (j < p.dims[1] && s_ok) ? (a - ytg) * f : 0.0f;
        if (s_ok) p.D[0][(int64_t)gs * NW + j] = d;
      } else if (s_ok && j < p.dims[1]) {
        p.out[(int64_t)gs * p.dims[1] + j] = a;
      }
    } else {
      hs[0][s][j] = a;
      if (TRAIN && s_ok) p.A[0][(int64_t)gs * NW + j] = a;
    }
  }
  __syncthreads();

  // ---- layers 2..L (padded units carry zeros, so every sum runs over 32)
#pragma unroll
  for (int l = 2; l <= NARROW_MAX_LAYERS; ++l) {
    if (l > p.L) break;
    const int dl = p.dims[l];
    float z = 0.0f;
#pragma unroll
    for (int i = 0; i < NW; ++i) z = fmaf(ws[l - 2][j][i], hs[cur][s][i], z);
    float a = 0.0f, f = 0.0f;
    if (j < dl) act_eval(p.acts[l - 1], z + bs[l - 1][j], a, f);
    fp[l - 1] = f;
    if (l == p.L) {
      if (TRAIN) {
        const float d = (j < dl && s_ok) ? (a - ytg) * f : 0.0f;
        hs[cur ^ 1][s][j] = d;
        if (s_ok) p.D[l - 1][(int64_t)gs * NW + j] = d;
      } else if (s_ok && j < dl) {
        p.out[(int64_t)gs * dl + j] = a;
      }
    } else {
      hs[cur ^ 1][s][j] = a;
      if (TRAIN && s_ok) p.A[l - 1][(int64_t)gs * NW + j] = a;
    }
    cur ^= 1;
    __syncthreads();
  }
  if (!TRAIN) return;

  // ---- hidden deltas, l = L-1 .. 1, with the weights W_{l+1} of this step
#pragma unroll
  for (int l = NARROW_MAX_LAYERS - 1; l >= 1; --l) {
    if (l >= p.L) continue;
    float t = 0.0f;
#pragma unroll
    for (int k = 0; k < NW; ++k) t = fmaf(ws[l - 1][k][j], hs[cur][s][k], t);
    const float d = j < p.dims[l] ? t * fp[l - 1] : 0.0f;
    hs[cur ^ 1][s][j] = d;
    if (s_ok) p.D[l - 1][(int64_t)gs * NW + j] = d;
    cur ^= 1;
    __syncthreads();
  }
}

// Workgroup = 8 waves, one (layer, 16-column tile, 16-unit half) over the whole
// batch: G[16 h + u][c0 + r] = sum over samples of delta[s][16 h + u] a_prev[s][c0 + r]
// on the 16x16x4 matrix cores.  Wave w takes every 8th group of 4 samples; the
// waves' sums are added in wave order, then the tile applies the SGD step.
constexpr int N2_WAVES = 8;
constexpr int N2_UNROLL = 32;  // groups of 4 samples loaded before use

__global__ void __launch_bounds__(N2_WAVES * 64) narrow_dw_kernel(const NarrowDwParams p) {
  __shared__ float red[N2_WAVES][16][17];
  __shared__ float bred[N2_WAVES][4][16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // consecutive workgroups land on different XCDs (round robin over 8); give
  // each XCD a contiguous run of tiles so that the two unit halves of a column
  // tile, and neighbouring column tiles, share the input rows in one L2
  const int nwg = p.tile_base[p.L];
  const int per = (nwg + 7) / 8;
  const int full = nwg - 8 * (per - 1);       // XCDs that get `per` tiles
  const int xcd = (int)blockIdx.x & 7, slot = (int)blockIdx.x >> 3;
  const int tile = xcd < full ? xcd * per + slot : full * per + (xcd - full) * (per - 1) + slot;
  int l = 0;
  while (l + 1 < p.L && tile >= p.tile_base[l + 1]) ++l;
  const int M = p.dims[l + 1], N = p.dims[l];
  const int nh = (M + 15) / 16;
  const int c = (tile - p.tile_base[l]) / nh, h = (tile - p.tile_base[l]) % nh;
  const int c0 = c * 16, u0 = h * 16;
  const float* xop = l == 0 ? p.X : p.A[l - 1];
  const int64_t ldx = l == 0 ? p.dims[0] : NARROW_WIDTH;
  const float* dl = p.D[l] + u0;

  const int r = lane & 15, g = lane >> 4;
  const bool col_ok = c0 + r < N;
  const float* xcol = xop + (col_ok ? c0 + r : 0);
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  float bsum = 0.0f;
  const int ngroups = (p.B + 3) / 4;
  for (int gb = wave; gb < ngroups; gb += N2_WAVES * N2_UNROLL) {
    float dv[N2_UNROLL], xv[N2_UNROLL];
#pragma unroll
    for (int u = 0; u < N2_UNROLL; ++u) {
      const int smp = (gb + u * N2_WAVES) * 4 + g;
      const int sc = smp < p.B ? smp : p.B - 1;
      dv[u] = dl[(int64_t)sc * NARROW_WIDTH + r];
      xv[u] = xcol[(int64_t)sc * ldx];
    }
#pragma unroll
    for (int u = 0; u < N2_UNROLL; ++u) {
      const bool ok = (gb + u * N2_WAVES) * 4 + g < p.B;
      const float a = ok ? dv[u] : 0.0f;
      const float b = (ok && col_ok) ? xv[u] : 0.0f;
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
      bsum += a;
    }
  }
  // accumulator register v of lane (r, g): unit u0 + 4 g + v, column c0 + r
#pragma unroll
  for (int v = 0; v < 4; ++v) red[wave][4 * g + v][r] = acc[v];
  if (c == 0) bred[wave][g][r] = bsum;
  __syncthreads();

  if (tid < 256) {
    const int i = tid >> 4, jj = tid & 15;   // unit within the half, column within the tile
    float gsum = red[0][i][jj];
#pragma unroll
    for (int w = 1; w < N2_WAVES; ++w) gsum += red[w][i][jj];
    if (u0 + i < M && c0 + jj < N) {
      const int64_t o = (int64_t)(u0 + i) * p.ldw[l] + c0 + jj;
      p.G[l][o] = gsum;
      p.W[l][o] = fmaf(-p.scale, gsum, p.Win[l][o]);
    }
  }
  if (c == 0 && tid < 16 && u0 + tid < M) {
    float gsum = 0.0f;
#pragma unroll
    for (int w = 0; w < N2_WAVES; ++w)
#pragma unroll
      for (int q = 0; q < 4; ++q) gsum = (w == 0 && q == 0) ? bred[0][0][tid] : gsum + bred[w][q][tid];
    p.gb[l][u0 + tid] = gsum;
    p.bias[l][u0 + tid] = fmaf(-p.scale, gsum, p.bin[l][u0 + tid]);
  }
}

hipError_t launch_narrow_fwd(bool train, const NarrowFwdParams& p, hipStream_t s) {
  const dim3 grid((p.B + NARROW_TILE - 1) / NARROW_TILE);
  if (train)
    narrow_fwd_kernel<true, N1_PRE_TRAIN><<<grid, N1_WAVES * 64, 0, s>>>(p);
  else
    narrow_fwd_kernel<false, N1_PRE_INFER><<<grid, N1_WAVES * 64, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_narrow_dw(const NarrowDwParams& p, hipStream_t s) {
  narrow_dw_kernel<<<dim3(p.tile_base[p.L]), N2_WAVES * 64, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace nf
