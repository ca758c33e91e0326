// Training step for narrow networks (every layer after the input has at most
// 32 units, like the paper's 784-30-10 MNIST network, section 4).
//
// Kernel 1, per tile of 4 samples (batches up to NARROW_SMALL_BATCH) or 16
// samples (larger batches), one workgroup of 8 waves:
//   layer 1   z_1 = W_1 x + b_1 on the fp32 matrix cores (4x4x1 blocks fed
//             from registers, or 16x16x4 with the input width staged through
//             LDS), the partial sums added in a fixed order;
//   layers 2+ one thread per (sample, unit) with the previous layer in LDS;
//   deltas    output delta (a_L - y) f'(z_L) and hidden deltas
//             (W_{l+1}^T delta_{l+1}) f'(z_l) (section 3.3), with f'(z_l) kept
//             in registers from the forward pass.
// Kernel 2, tendencies of every layer (sections 3.3-3.5): workgroup
//   (layer, 16-column tile, 16-unit half) forms the batch sum of delta (outer)
//   activation for its block on the matrix cores (16x16x4), its 8 waves
//   splitting the batch and their sums added in wave order; it then stores
//   the tendency and writes W' = W - (eta/B) G itself (into the other
//   parameter buffer), so no workgroup waits on another.
// The order of every sum is fixed, so results are reproducible bit for bit.
#include <type_traits>

#include "nf_act.h"
#include "nf_internal.h"

namespace nf {

typedef float floatx4 __attribute__((ext_vector_type(4)));

// v if c, else zeros; written per component (a conditional on the vector
// type itself is lowered through private memory)
__device__ __forceinline__ float4 keep_if(bool c, float4 v) {
  return make_float4(c ? v.x : 0.0f, c ? v.y : 0.0f, c ? v.z : 0.0f, c ? v.w : 0.0f);
}

// The float4 of lane src_byte / 4, by one backward permute per dword.  The
// vector memory pipeline takes a 16-byte load at full rate only when each
// quad of lanes (4 consecutive lanes) reads 64 consecutive bytes; where the
// lanes of a quad read four different rows, as the matrix-core operand
// layouts would have them, it delivers about a third of that.  So inputs are
// loaded quad-contiguous and moved across lanes to the operand layout.
__device__ __forceinline__ float4 lane_permute4(int src_byte, float4 v) {
  float4 o;
  o.x = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src_byte, __builtin_bit_cast(int, v.x)));
  o.y = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src_byte, __builtin_bit_cast(int, v.y)));
  o.z = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src_byte, __builtin_bit_cast(int, v.z)));
  o.w = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src_byte, __builtin_bit_cast(int, v.w)));
  return o;
}

// A buffer offset past every range the narrow kernels read through buffer
// resources: a load there returns zeros without touching memory.
constexpr unsigned NB_OOB = NARROW_OOB;

constexpr int N1_WAVES = 8;
constexpr int N1_KC = 16 * N1_WAVES;  // inputs per LDS stage: one 16-wide group per wave
constexpr int N1_KP = N1_KC + 4;      // padded LDS row
// chunks requested together: 8 for training (one launch of few workgroups),
// 4 for inference (fewer registers, two workgroups per CU)
constexpr int N1_PRE_TRAIN = 8;
constexpr int N1_PRE_INFER = 4;

// The weights of layers 2..L, staged in LDS by every tile (the per-sample
// threads read them again and again), and every layer's bias for unit tid % 32
// (the unit the thread handles in the tail, so the biases stay in registers).
// Each thread loads its share before layer 1 and stores the weights to LDS
// afterwards, so the loads land while layer 1 runs.
constexpr int NSTAGE = NARROW_WIDTH * NARROW_WIDTH / (N1_WAVES * 64);
static_assert(NARROW_WIDTH * NARROW_WIDTH % (N1_WAVES * 64) == 0, "staging split");

struct SmallLayers {
  float w[NARROW_MAX_LAYERS - 1][NSTAGE];
  float b[NARROW_MAX_LAYERS];
};

// The layer loops are unrolled so that every kernel-argument index is a
// constant, and the loads carry no conditions: the padded layout (zeros past
// the layer sizes, a zero block past the last layer) makes every entry of the
// 32 x 32 blocks readable, so all the loads issue together at kernel start.
__device__ __forceinline__ void load_small_layers(const NarrowFwdParams& p, int tid,
                                                  SmallLayers& r) {
#pragma unroll
  for (int li = 0; li < NARROW_MAX_LAYERS - 1; ++li)
#pragma unroll
    for (int u = 0; u < NSTAGE; ++u) r.w[li][u] = p.W[li + 1][tid + u * N1_WAVES * 64];
#pragma unroll
  for (int l = 0; l < NARROW_MAX_LAYERS; ++l) r.b[l] = p.bias[l][tid & (NARROW_WIDTH - 1)];
}

// LDS row pitch of the per-sample activations and the small layers' weights:
// 16-byte aligned rows, so a row is read with eight 16-byte loads.
constexpr int NWP = NARROW_WIDTH + 4;

// The small layers' weights go to LDS twice when training: ws[l][j][i] = W(j, i)
// for the forward sums and wsT[l][i][j] = W(j, i) for the delta sums, so
// both read whole rows.
template <bool TRANSPOSED>
__device__ __forceinline__ void store_small_layers(const SmallLayers& r, int tid,
                                                   float (*ws)[NARROW_WIDTH][NWP],
                                                   float (*wsT)[NARROW_WIDTH][NWP]) {
  constexpr int NW = NARROW_WIDTH;
#pragma unroll
  for (int li = 0; li < NARROW_MAX_LAYERS - 1; ++li)
#pragma unroll
    for (int u = 0; u < NSTAGE; ++u) {
      const int e = tid + u * N1_WAVES * 64;
      ws[li][e / NW][e % NW] = r.w[li][u];
      if (TRANSPOSED) wsT[li][e % NW][e / NW] = r.w[li][u];
    }
}

// sum over i < 32 of w[i] h[i] from two 16-byte aligned LDS rows, in four
// interleaved partial sums added pairwise
__device__ __forceinline__ float dot32(const float* w, const float* h) {
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int m = 0; m < NARROW_WIDTH / 4; ++m) {
    const float4 a = *reinterpret_cast<const float4*>(w + 4 * m);
    const float4 x = *reinterpret_cast<const float4*>(h + 4 * m);
    acc[0] = fmaf(a.x, x.x, acc[0]);
    acc[1] = fmaf(a.y, x.y, acc[1]);
    acc[2] = fmaf(a.z, x.z, acc[2]);
    acc[3] = fmaf(a.w, x.w, acc[3]);
  }
  return (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

// Target of thread (sample tid / 32, output unit tid % 32) of a T-sample tile.
template <int T>
__device__ __forceinline__ float load_target(const NarrowFwdParams& p, int s0, int tid) {
  // read from a clamped (always valid) position without a branch, so the
  // load issues with the others at kernel start
  const int ys = s0 + (tid >> 5), yu = tid & 31;
  const bool ok = tid < T * NARROW_WIDTH && ys < p.B && yu < p.dout;
  const int yr = ys < p.B ? ys : p.B - 1, yc = yu < p.dout ? yu : p.dout - 1;
  const float v = p.Y[(int64_t)yr * p.dout + yc];
  return ok ? v : 0.0f;
}

// The tail's thread (s, j) = (tid / 32, tid % 32) keeps each sample's 32 units
// in one wave, so every phase of the tail reads only what its own wave wrote
// in the phase before: LDS operations of a wave complete in order, and a
// wavefront-scope fence keeps the compiler from moving them across the
// boundary.  The persistent inference kernel (BLOCK) still needs workgroup
// barriers: it reuses the layer-1 sums and the staged outputs across waves.
template <bool BLOCK>
__device__ __forceinline__ void tail_sync() {
  if constexpr (BLOCK) {
    __syncthreads();
  } else {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// Everything after the layer-1 sums, for thread (s, j) = (tid / 32, tid % 32):
// sample s of the T-sample tile, unit j of the current layer.  Layer 1's
// activation, layers 2..L with the previous layer in LDS (padded units carry
// zeros, so every sum runs over 32), the output delta (a_L - y) f'(z_L) and
// the hidden deltas (W_{l+1}^T delta_{l+1}) f'(z_l) (section 3.3) with
// f'(z_l) kept in registers.  Threads past 32 T only join the workgroup
// barriers of the inference kernel.
// Inference writes f(z_L) to the output, or with STAGED to ostage[s][j] in LDS.
template <bool TRAIN, int T, bool STAGED = false>
__device__ __forceinline__ void narrow_tail(const NarrowFwdParams& p, int s0, int tid, float z1,
                                            float ytg, float (*hs)[T][NWP],
                                            const float (*ws)[NARROW_WIDTH][NWP],
                                            const float (*wsT)[NARROW_WIDTH][NWP],
                                            const float (&bias)[NARROW_MAX_LAYERS],
                                            float (*ostage)[NARROW_WIDTH] = nullptr) {
  constexpr int NW = NARROW_WIDTH;
  const bool active = tid < T * NW;
  const int s = active ? tid >> 5 : 0, j = tid & 31;
  const int gs = s0 + s;
  const bool s_ok = active && gs < p.B;
  float fp[NARROW_MAX_LAYERS];
#pragma unroll
  for (int l = 0; l < NARROW_MAX_LAYERS; ++l) fp[l] = 0.0f;
  int cur = 0;
  if (active) {
    float a = 0.0f, f = 0.0f;
    if (j < p.dims[1]) act_eval(p.acts[0], z1 + bias[0], a, f);
    fp[0] = f;
    if (p.L == 1) {
      if (TRAIN) {
        const float d = (j < p.dims[1] && s_ok) ? (a - ytg) * f : 0.0f;
        if (s_ok) p.D[0][(int64_t)gs * NW + j] = d;
      } else if (STAGED) {
        ostage[s][j] = a;
      } else if (s_ok && j < p.dims[1]) {
        p.out[(int64_t)gs * p.dims[1] + j] = a;
      }
    } else {
      hs[0][s][j] = a;
      if (TRAIN && s_ok) p.A[0][(int64_t)gs * NW + j] = a;
    }
  }
  tail_sync<STAGED>();

  // ---- layers 2..L
#pragma unroll
  for (int l = 2; l <= NARROW_MAX_LAYERS; ++l) {
    if (l > p.L) break;
    if (active) {
      const int dl = p.dims[l];
      const float z = dot32(ws[l - 2][j], hs[cur][s]);
      float a = 0.0f, f = 0.0f;
      if (j < dl) act_eval(p.acts[l - 1], z + bias[l - 1], a, f);
      fp[l - 1] = f;
      if (l == p.L) {
        if (TRAIN) {
          const float d = (j < dl && s_ok) ? (a - ytg) * f : 0.0f;
          hs[cur ^ 1][s][j] = d;
          if (s_ok) p.D[l - 1][(int64_t)gs * NW + j] = d;
        } else if (STAGED) {
          ostage[s][j] = a;
        } else if (s_ok && j < dl) {
          p.out[(int64_t)gs * dl + j] = a;
        }
      } else {
        hs[cur ^ 1][s][j] = a;
        if (TRAIN && s_ok) p.A[l - 1][(int64_t)gs * NW + j] = a;
      }
    }
    cur ^= 1;
    tail_sync<STAGED>();
  }
  if (!TRAIN) return;

  // ---- hidden deltas, l = L-1 .. 1, with the weights W_{l+1} of this step
  // (layer 1's delta is read by no later phase: no LDS copy, no barrier)
#pragma unroll
  for (int l = NARROW_MAX_LAYERS - 1; l >= 1; --l) {
    if (l >= p.L) continue;
    if (active) {
      const float t = dot32(wsT[l - 1][j], hs[cur][s]);
      const float d = j < p.dims[l] ? t * fp[l - 1] : 0.0f;
      if (l > 1) hs[cur ^ 1][s][j] = d;
      if (s_ok) p.D[l - 1][(int64_t)gs * NW + j] = d;
    }
    cur ^= 1;
    if (l > 1) tail_sync<STAGED>();
  }
}

// ---------------------------------------------------------------------------
// 16-sample tiles (large batches): layer 1 on the 16x16x4 matrix cores, the
// input width staged through LDS in 128-wide chunks.
// ---------------------------------------------------------------------------
template <bool TRAIN, int N1_PRE>
__global__ void __launch_bounds__(N1_WAVES * 64) narrow_fwd16_kernel(const NarrowFwdParams p) {
  constexpr int T = NARROW_TILE;
  constexpr int NW = NARROW_WIDTH;
  // layer-1 staging (input chunk xs, W_1 chunk wsl, two buffers each); the
  // per-wave partial sums zp reuse the same bytes once layer 1 is done
  __shared__ __attribute__((aligned(16))) float stage[2 * (T + NW) * N1_KP];
  static_assert(N1_WAVES * T * (NW + 1) <= 2 * (T + NW) * N1_KP, "zp must fit the staging area");
  auto xs = reinterpret_cast<float(*)[T][N1_KP]>(stage);
  auto wsl = reinterpret_cast<float(*)[NW][N1_KP]>(stage + 2 * T * N1_KP);
  auto zp = reinterpret_cast<float(*)[T][NW + 1]>(stage);
  __shared__ __attribute__((aligned(16))) float hs[2][T][NWP];   // activations, then deltas
  __shared__ __attribute__((aligned(16))) float ws[NARROW_MAX_LAYERS - 1][NW][NWP];  // W_2 .. W_L
  __shared__ __attribute__((aligned(16))) float wsT[TRAIN ? NARROW_MAX_LAYERS - 1 : 1][NW][NWP];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int s0 = blockIdx.x * T;

  SmallLayers sl;
  load_small_layers(p, tid, sl);
  const float ytg = TRAIN ? load_target<T>(p, s0, tid) : 0.0f;

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
    const int nch = (p.d0 + N1_KC - 1) / N1_KC;
    // this thread's share of a chunk: one float4 of X, two of W_1 (whose
    // rows are padded to 32 with zeros)
    const int xrow = tid / (N1_KC / 4), xq = tid % (N1_KC / 4);
    const bool xrow_ok = s0 + xrow < p.B;
    const float* xsrc = p.X + (int64_t)(xrow_ok ? s0 + xrow : p.B - 1) * p.d0;
    const float* wsrc0 = p.W[0] + (int64_t)xrow * p.ldw[0];
    const float* wsrc1 = p.W[0] + (int64_t)(16 + xrow) * p.ldw[0];
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
        wr0[u] = keep_if(k_ok, w0);
        wr1[u] = keep_if(k_ok, w1);
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
  store_small_layers<TRAIN>(sl, tid, ws, wsT);
  __syncthreads();

  // z_1 of (sample tid / 32, unit tid % 32): the waves' sums in wave order
  float z1;
  {
    const int s = tid >> 5, j = tid & 31;
    z1 = zp[0][s][j];
#pragma unroll
    for (int w = 1; w < N1_WAVES; ++w) z1 += zp[w][s][j];
  }
  narrow_tail<TRAIN, T>(p, s0, tid, z1, ytg, hs, ws, wsT, sl.b);
}

// ---------------------------------------------------------------------------
// 4-sample tiles (training batches of up to NARROW_SMALL_BATCH samples: a
// 1000-sample batch is 250 workgroups, one per CU, instead of 63).  Layer 1 on
// the 4x4x1 matrix cores straight from registers: each instruction forms 16
// independent 4x4 blocks (4 samples x 4 units), and the 16 blocks take 16
// different inputs, so one instruction covers 4 samples x 4 units x 16 inputs.
// Lane (b, q) = (lane / 4, lane % 4) loads one float4 of its sample row q and
// one float4 of W_1 row 4 ug + q (for each of the 8 unit groups ug) at inputs
// 64 t + 4 b .. 64 t + 4 b + 3 of step t; the four components feed four
// MFMAs.  Wave w takes steps w, w + 8, ...  The (wave, block) partial sums of
// every (sample, unit) are then added in LDS in a fixed order.
// ---------------------------------------------------------------------------
constexpr int N4_T = 4;                      // samples per workgroup
constexpr int N4_KS = 64;                    // inputs per step
constexpr int N4_UG = NARROW_WIDTH / 4;      // unit groups
constexpr int N4_PRE = 2;                    // steps per wave requested together
constexpr int N4_PARTS = N1_WAVES * 16;      // (wave, block) partial sums per output
constexpr int N4_RP = 36;                    // padded row: conflict-free stores
constexpr int N4_SS = N4_PARTS * N4_RP + 32; // sample stride (other bank half)
static_assert(N1_WAVES * 64 == 4 * N4_T * NARROW_WIDTH, "four partial sums per output");

template <bool TRAIN>
__global__ void __launch_bounds__(N1_WAVES * 64) narrow_fwd4_kernel(const NarrowFwdParams p) {
  constexpr int T = N4_T;
  constexpr int NW = NARROW_WIDTH;
  __shared__ float red[T * N4_SS];                           // [sample][wave*16+block][unit]
  __shared__ float psum[4][T][NW];
  __shared__ __attribute__((aligned(16))) float hs[2][T][NWP];
  __shared__ __attribute__((aligned(16))) float ws[NARROW_MAX_LAYERS - 1][NW][NWP];
  __shared__ __attribute__((aligned(16))) float wsT[TRAIN ? NARROW_MAX_LAYERS - 1 : 1][NW][NWP];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int s0 = blockIdx.x * T;

  SmallLayers sl;
  load_small_layers(p, tid, sl);
  const float ytg = TRAIN ? load_target<T>(p, s0, tid) : 0.0f;

  {
    const int b = lane >> 2, q = lane & 3;
    // the tile's input rows through a buffer resource that ends at the last
    // row, and W_1 packed in this kernel's operand layout (W1f: lane 4 b + q
    // of block (t, ug) holds W_1[4 ug + q][64 t + 4 b ..], one contiguous 1 KiB
    // per instruction); rows past the batch, inputs past the width and steps
    // past the last (given an offset past the end) read as zeros without a
    // memory access, so no bytes go to loads whose values are not used.  The
    // inputs are loaded with lane 16 qx + bx taking sample qx, inputs
    // 64 t + 4 bx .. (each quad of lanes 64 consecutive bytes, which the vector
    // memory pipeline takes at full rate) and moved to the operand layout
    // (lane 4 b + q: sample q, inputs 64 t + 4 b ..) by a backward permute.
    const int qx = lane >> 4, bx = lane & 15;
    const int src_byte = 4 * (16 * q + b);
    const int nrows = p.B - s0 < T ? p.B - s0 : T;
    const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(p.X + (int64_t)s0 * p.d0), (short)0, nrows * p.d0 * 4, 0x00020000);
    const int nsteps = (p.d0 + N4_KS - 1) / N4_KS;
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        (void*)p.W1f, (short)0, nsteps * NARROW_PACK_W1F_BLOCK * 4, 0x00020000);
    floatx4 acc[N4_UG];
#pragma unroll
    for (int ug = 0; ug < N4_UG; ++ug) acc[ug] = floatx4{0.f, 0.f, 0.f, 0.f};
    // workgroups start at different steps (rotated by the tile index), so the
    // workgroups that start together do not all ask for the same W_1 lines
    const int rot = (int)(blockIdx.x % (unsigned)nsteps);
    // the first block runs unconditionally (a wave without steps adds zeros),
    // so its loads are not held behind a branch
    int t0 = wave;
    do {
      // all loads of the block first; inputs past the width load as zeros
      // (the width is a multiple of 4, so a float4 is wholly in or out)
      float4 xr[N4_PRE], wr[N4_PRE][N4_UG];
#pragma unroll
      for (int u = 0; u < N4_PRE; ++u) {
        int t = t0 + u * N1_WAVES;
        const bool tin = t < nsteps;
        if (tin) t = t + rot < nsteps ? t + rot : t + rot - nsteps;
        const int kx = t * N4_KS + 4 * bx;
        const bool okx = tin && kx < p.d0;
        xr[u] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(
                                               xres, okx ? 4 * (qx * p.d0 + kx) : (int)NB_OOB, 0, 0));
#pragma unroll
        for (int ug = 0; ug < N4_UG; ++ug)
          wr[u][ug] = __builtin_bit_cast(
              float4, __builtin_amdgcn_raw_buffer_load_b128(
                          wres, tin ? 16 * ((t * 8 + ug) * 64 + lane) : (int)NB_OOB, 0, 0));
      }
      // keep every load of the block ahead of the first matrix instruction
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < N4_PRE; ++u) xr[u] = lane_permute4(src_byte, xr[u]);
#pragma unroll
      for (int u = 0; u < N4_PRE; ++u) {
#pragma unroll
        for (int ug = 0; ug < N4_UG; ++ug)
          acc[ug] = __builtin_amdgcn_mfma_f32_4x4x1f32(xr[u].x, wr[u][ug].x, acc[ug], 0, 0, 0);
#pragma unroll
        for (int ug = 0; ug < N4_UG; ++ug)
          acc[ug] = __builtin_amdgcn_mfma_f32_4x4x1f32(xr[u].y, wr[u][ug].y, acc[ug], 0, 0, 0);
#pragma unroll
        for (int ug = 0; ug < N4_UG; ++ug)
          acc[ug] = __builtin_amdgcn_mfma_f32_4x4x1f32(xr[u].z, wr[u][ug].z, acc[ug], 0, 0, 0);
#pragma unroll
        for (int ug = 0; ug < N4_UG; ++ug)
          acc[ug] = __builtin_amdgcn_mfma_f32_4x4x1f32(xr[u].w, wr[u][ug].w, acc[ug], 0, 0, 0);
      }
      t0 += N1_WAVES * N4_PRE;
    } while (t0 < nsteps);
    // accumulator register v of lane (b, q): block b's sum for sample v, unit 4 ug + q
#pragma unroll
    for (int ug = 0; ug < N4_UG; ++ug)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        red[v * N4_SS + (wave * 16 + b) * N4_RP + 4 * ug + q] = acc[ug][v];
  }
  store_small_layers<TRAIN>(sl, tid, ws, wsT);
  __syncthreads();

  // every thread adds a quarter of the (wave, block) sums of one output, in
  // order; the quarters are then added pairwise
  {
    const int part = tid >> 7, s = (tid >> 5) & 3, j = tid & 31;
    const float* src = red + s * N4_SS + part * (N4_PARTS / 4) * N4_RP + j;
    float t = src[0];
#pragma unroll
    for (int r = 1; r < N4_PARTS / 4; ++r) t += src[r * N4_RP];
    psum[part][s][j] = t;
  }
  __syncthreads();
  float z1 = 0.0f;
  if (tid < T * NW) {
    const int s = tid >> 5, j = tid & 31;
    z1 = (psum[0][s][j] + psum[1][s][j]) + (psum[2][s][j] + psum[3][s][j]);
  }
  narrow_tail<TRAIN, T>(p, s0, tid, z1, ytg, hs, ws, wsT, sl.b);
}

// one of four per-layer arguments, picked by value (so that an argument load
// does not wait on the index)
template <class V>
__device__ __forceinline__ V pick(int l, V a0, V a1, V a2, V a3) {
  return l == 0 ? a0 : (l == 1 ? a1 : (l == 2 ? a2 : a3));
}

// ---------------------------------------------------------------------------
// Inference over large batches.  One persistent workgroup of 8 waves per CU
// walks a contiguous, balanced run of 16-sample tiles; every wave does both
// parts of the work.
//
// Layer 1: W_1 stays in the waves' registers for the whole launch, the wave
// of chunk group q holding the 16-wide input chunks q, q + 8, ... of all 32
// units (a CU reads W_1 once, from its packed copy in the operand layout, a
// contiguous KiB per load, requested before any input: a CU keeps a bounded
// number of loads in flight and they complete in order, so W_1 behind inputs
// from HBM would arrive only at the inputs' pace); the groups are dealt to the waves rotated by
// the workgroup index, so the workgroups that start together ask for
// different lines of W_1 first.  Layer 1 runs as z^T = W_1 x^T on the
// 16x16x4 matrix instruction, units as rows and samples as columns; each
// wave leaves its partial sums of a tile in one of NI_NB LDS buffers and
// counts them there.  The inputs of later tiles are requested before the
// matrix work of the current one, through a buffer resource: rows past the
// batch and inputs past the width come back as zeros without touching
// memory, so every load is unconditional.
//
// The rest of the network, one tile behind: wave w takes samples 2w and
// 2w + 1 of the tile, lane (s, u) = (lane / 32, lane % 32) unit u of one of
// them.  It adds the 8 partial sums in group order, adds the bias and applies
// f, then runs each later layer as a 32-term dot product over the previous
// layer's values of its sample (a per-wave LDS row) with the weights in LDS.
// One value per lane keeps the dependent instruction chains of the
// activations short and spreads them over all SIMDs; running a tile late
// lets a wave start the next tile without waiting for the slowest wave.  The
// outputs collect in LDS and are written every NI_OUT tiles and at the end:
// a store in flight would make every later use of a prefetched input wait
// for all outstanding loads (loads and stores share one wait counter).
//
// Counters in LDS: zst[b] counts the partial-sum stores into buffer b and
// zrd[b] the waves that have read it, each growing by 8 per use of the
// buffer.  A wave writes tile t into buffer t % NI_NB once all 8 have read
// tile t - NI_NB from it, and reads tile t once all 8 have stored it.  A
// wave's LDS operations complete in order; counts are release additions after
// the accesses they cover, and waits are acquire loads polled with a short
// sleep.  Every wait is bounded (NI_SPIN polls): correct code never comes
// near the bound, and a wave that reached it would go on rather than hang.
// ---------------------------------------------------------------------------
constexpr int NI_CH = 16;                  // inputs per chunk: a float4 per lane group
constexpr int NI_SLOTS = 3;                // tiles of inputs held: the current one + two ahead
constexpr int NI_QWAIT = 7;                // loads of the current tile left in flight when the next is requested
constexpr int NI_MW = N1_WAVES;            // chunk groups: one per wave
constexpr int NI_NB = 3;                   // partial-sum buffers
constexpr int NI_ZS = NARROW_TILE + 1;     // partial-sum row stride: conflict-free reads
constexpr int NI_OUT = 16;                 // tiles of outputs held before they are written
constexpr unsigned NI_OOB = NB_OOB;
constexpr int NI_SPIN = 1 << 22;           // polls before a wait gives up (about 0.1 s)
static_assert(2 * N1_WAVES == NARROW_TILE, "two samples of a tile per wave");

// waits until at most N of the wave's vector memory operations are in flight
// (they complete in order, so the oldest ones have landed)
template <int N>
__device__ __forceinline__ void ni_wait_loads() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// waits until the LDS counter c reaches at least v (acquire), at most NI_SPIN polls
__device__ __forceinline__ void ni_wait_at_least(unsigned* c, unsigned v) {
  for (int k = 0; k < NI_SPIN; ++k) {
    if (__hip_atomic_load(c, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) >= v) return;
    __builtin_amdgcn_s_sleep(1);
  }
}

__device__ __forceinline__ float ni_act(int act, float z) {
  float f, fp;
  act_eval(act, z, f, fp);
  return f;
}

template <int MC, int NS = NI_SLOTS, int NQ = NI_QWAIT>
__global__ void __launch_bounds__(N1_WAVES * 64) narrow_infer_kernel(const NarrowFwdParams p) {
  static_assert(NS == 2 || NS == 3, "two or three input slots");
  static_assert(NQ >= 0, "loads left in flight");
  constexpr int Q = NQ < MC ? NQ : MC;
  constexpr int T = NARROW_TILE;
  constexpr int NW = NARROW_WIDTH;
  // layer-1 partial sums [buffer][chunk group][unit][sample]
  __shared__ float zq[NI_NB][NI_MW][NW][NI_ZS];
  __shared__ unsigned zst[NI_NB], zrd[NI_NB];
  __shared__ __attribute__((aligned(16))) float ws[NARROW_MAX_LAYERS - 1][NW][NWP];
  __shared__ float bs[NARROW_MAX_LAYERS][NW];
  // a layer's values of each wave's two samples, and the outputs held
  __shared__ __attribute__((aligned(16))) float hs[N1_WAVES][2][NWP];
  __shared__ float os[N1_WAVES][NI_OUT][2][NW];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, g = lane >> 4;

  // this workgroup's tiles [t0, t1): a contiguous, balanced share
  const int ntiles = (p.B + T - 1) / T;
  const int t0 = (int)((int64_t)blockIdx.x * ntiles / gridDim.x);
  const int t1 = (int)((int64_t)(blockIdx.x + 1) * ntiles / gridDim.x);
  const int nt = t1 - t0;
  if (tid < NI_NB) {
    zst[tid] = 0u;
    zrd[tid] = 0u;
  }
  __syncthreads();

  // the small layers' weights and every bias: requested first and staged in
  // LDS once the big loads are issued (a store waits for its load, and loads
  // complete in order); each wave stages its share before it counts its first
  // tile, and a wave reads them only after every wave has counted that tile.
  // Every entry of the padded 32 x 32 blocks is readable, so the loads are
  // unconditional (clamped indices).
  constexpr int NSMALL = (NW * NW + N1_WAVES * 64 - 1) / (N1_WAVES * 64);
  float wv[NARROW_MAX_LAYERS - 1][NSMALL];
#pragma unroll
  for (int li = 0; li < NARROW_MAX_LAYERS - 1; ++li)
#pragma unroll
    for (int u = 0; u < NSMALL; ++u) {
      const int e = tid + u * N1_WAVES * 64;
      wv[li][u] = p.W[li + 1][e < NW * NW ? e : NW * NW - 1];
    }
  const int bl = (tid >> 5) & (NARROW_MAX_LAYERS - 1);
  const float bv = pick(bl, p.bias[0], p.bias[1], p.bias[2], p.bias[3])[tid & (NW - 1)];
  // issued before every later load, so that staging them waits for them alone
  __builtin_amdgcn_sched_barrier(0);
  const int nch = (p.d0 + NI_CH - 1) / NI_CH;
  const int grp = (int)((wave + blockIdx.x) % NI_MW);
  // chunks of this group: MC or MC - 1 (MC is the launch's ceil(nch / NI_MW))
  const bool last_mine = (grp + NI_MW * (MC - 1)) < nch;
  // lane (r, g) feeds unit r (and 16 + r) and sample r with inputs 16 c + 4 g
  // .. 16 c + 4 g + 3 of chunk c = grp + NI_MW i, one per instruction; it
  // loads the inputs of row m = lane / 4 and group e = lane % 4 and takes its
  // own from lane 4 r + g.  Chunks i < MC - 1 lie wholly inside the input
  // width; the last one may be partial or absent, and its inputs past the
  // width are read at an offset past the buffer.
  const int m = lane >> 2, e = lane & 3;
  const int src_byte = 4 * (4 * r + g);
  const unsigned kofs = 4u * (unsigned)(grp * NI_CH + 4 * e);
  const int klast = (grp + NI_MW * (MC - 1)) * NI_CH + 4 * e;
  const unsigned kofs_last = klast < p.d0 ? 4u * (unsigned)klast : NI_OOB;
  auto koff = [&](int i) {
    return i < MC - 1 ? kofs + 4u * NI_MW * NI_CH * i : kofs_last;
  };
  // W_1 packed in this kernel's operand layout (W1i: lane r + 16 g of block
  // (c, h) holds W_1[16 h + r][16 c + 4 g ..]): one contiguous 1 KiB per
  // instruction, no permute; chunks past the last read as zeros
  const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
      (void*)p.W1i, (short)0, nch * NARROW_PACK_W1I_BLOCK * 4, 0x00020000);
  auto wload = [&](int i, int h) {
    const int c = grp + NI_MW * i;
    const unsigned off = c < nch ? 16u * (unsigned)((2 * c + h) * 64 + lane) : NI_OOB;
    return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(wres, off, 0, 0));
  };
  // the rows of this workgroup's tiles (fewer than NI_OOB bytes: the host
  // picks another kernel otherwise)
  const int row0 = t0 * T;
  const int nrows = (p.B < t1 * T ? p.B : t1 * T) - row0;
  const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.X + (int64_t)row0 * p.d0), (short)0, nrows * p.d0 * 4, 0x00020000);
  auto xload = [&](int tt, int i) {
    const unsigned roff = 4u * (unsigned)((tt * T + m) * p.d0);
    return __builtin_bit_cast(
        float4, __builtin_amdgcn_raw_buffer_load_b128(xres, roff + koff(i), 0, 0));
  };
  auto load_tile = [&](float4(&dst)[MC], int tt) {
#pragma unroll
    for (int i = 0; i < MC; ++i) dst[i] = xload(tt, i);
  };
  float4 wlo[MC], whi[MC];
  float4 x[NS][MC];
#pragma unroll
  for (int i = 0; i < MC; ++i) {
    wlo[i] = wload(i, 0);
    whi[i] = wload(i, 1);
  }
  load_tile(x[0], 0);
  if constexpr (NS == 3) load_tile(x[1], 1);
  // every load of the prologue is issued before the first wait
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int li = 0; li < NARROW_MAX_LAYERS - 1; ++li)
#pragma unroll
    for (int u = 0; u < NSMALL; ++u) {
      const int e2 = tid + u * N1_WAVES * 64;
      if (e2 < NW * NW) ws[li][e2 / NW][e2 % NW] = wv[li][u];
    }
  if (tid < NARROW_MAX_LAYERS * NW) bs[bl][tid & (NW - 1)] = bv;

  // layer 1 of tile tt from its inputs xc; the partial sums go to buffer
  // tt % NI_NB once every wave has read the tile that used it before
  auto tile = [&](const float4(&xc)[MC], int tt) {
    floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < MC; ++i) {
      if (i < MC - 1 || last_mine) {
        const float4 v = lane_permute4(src_byte, xc[i]);
        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(wlo[i].x, v.x, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(whi[i].x, v.x, acc1, 0, 0, 0);
        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(wlo[i].y, v.y, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(whi[i].y, v.y, acc1, 0, 0, 0);
        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(wlo[i].z, v.z, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(whi[i].z, v.z, acc1, 0, 0, 0);
        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(wlo[i].w, v.w, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(whi[i].w, v.w, acc1, 0, 0, 0);
      }
    }
    const int b = tt % NI_NB;
    if (tt >= NI_NB) ni_wait_at_least(&zrd[b], (unsigned)(NI_MW * (tt / NI_NB)));
    // accumulator register v: unit 4 g + v (+ 16) of sample r
    float* zrow = &zq[b][grp][4 * g][r];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      zrow[v * NI_ZS] = acc0[v];
      zrow[(16 + v) * NI_ZS] = acc1[v];
    }
    if (lane == 0) __hip_atomic_fetch_add(&zst[b], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
  };

  // layers 1 (the rest of it) to L for this wave's two samples of tile tt
  const int sl = lane >> 5, u = lane & (NW - 1);
  const int js = 2 * wave + sl;  // sample within the tile
  auto flush = [&](int tt) {     // outputs of tiles (tt / NI_OUT) * NI_OUT .. tt
    const int tf = tt - tt % NI_OUT;
    for (int q = tf; q <= tt; ++q) {
      const int smp = (t0 + q) * T + js;
      if (u < p.dout && smp < p.B) p.out[(int64_t)smp * p.dout + u] = os[wave][q % NI_OUT][sl][u];
    }
  };
  auto rest = [&](int tt) {
    const int b = tt % NI_NB;
    ni_wait_at_least(&zst[b], (unsigned)(NI_MW * (tt / NI_NB + 1)));
    float z = zq[b][0][u][js];
#pragma unroll
    for (int q = 1; q < NI_MW; ++q) z += zq[b][q][u][js];
    if (lane == 0) __hip_atomic_fetch_add(&zrd[b], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    float h = ni_act(p.acts[0], z + bs[0][u]);
    for (int l = 2; l <= p.L; ++l) {
      hs[wave][sl][u] = h;
      const float* wr = &ws[l - 2][u][0];
      const float* hr = &hs[wave][sl][0];
      float a0 = bs[l - 1][u], a1 = 0.0f;
#pragma unroll
      for (int k = 0; k < NW; k += 8) {
        const float4 w0 = *reinterpret_cast<const float4*>(wr + k);
        const float4 h0 = *reinterpret_cast<const float4*>(hr + k);
        const float4 w1 = *reinterpret_cast<const float4*>(wr + k + 4);
        const float4 h1 = *reinterpret_cast<const float4*>(hr + k + 4);
        a0 = fmaf(w0.x, h0.x, a0);
        a1 = fmaf(w1.x, h1.x, a1);
        a0 = fmaf(w0.y, h0.y, a0);
        a1 = fmaf(w1.y, h1.y, a1);
        a0 = fmaf(w0.z, h0.z, a0);
        a1 = fmaf(w1.z, h1.z, a1);
        a0 = fmaf(w0.w, h0.w, a0);
        a1 = fmaf(w1.w, h1.w, a1);
      }
      h = ni_act(pick(l - 1, p.acts[0], p.acts[1], p.acts[2], p.acts[3]), a0 + a1);
    }
    os[wave][tt % NI_OUT][sl][u] = h;
    if (tt % NI_OUT == NI_OUT - 1 || tt == nt - 1) flush(tt);
  };

  // Tile tt is in slot tt % NS.  Before its matrix work a wave requests the
  // inputs of tile tt + NS - 1 (past the last tile: zeros, no traffic), once
  // at most Q loads of tile tt are still in flight; after it, the wave
  // finishes tile tt - 1.  The loop runs whole groups of NS tiles (slot
  // indices must be constants); the last tiles follow it, their inputs
  // already requested.
  auto step = [&](auto cur, auto nxt, int tt) {
    ni_wait_loads<Q + (NS - 2) * MC>();
    __builtin_amdgcn_sched_barrier(0);
    load_tile(x[decltype(nxt)::value], tt + NS - 1);
    __builtin_amdgcn_sched_barrier(0);
    tile(x[decltype(cur)::value], tt);
    if (tt > 0) rest(tt - 1);
  };
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;
  int tb = 0;
  if constexpr (NS == 2) {
    for (; tb + 2 <= nt; tb += 2) {
      step(S0{}, S1{}, tb);
      step(S1{}, S0{}, tb + 1);
    }
    if (tb < nt) {
      tile(x[0], tb);
      if (tb > 0) rest(tb - 1);
    }
  } else {
    for (; tb + 3 <= nt; tb += 3) {
      step(S0{}, S2{}, tb);
      step(S1{}, S0{}, tb + 1);
      step(S2{}, S1{}, tb + 2);
    }
    if (tb < nt) {
      tile(x[0], tb);
      if (tb > 0) rest(tb - 1);
    }
    if (tb + 1 < nt) {
      tile(x[1], tb + 1);
      rest(tb);
    }
  }
  if (nt > 0) rest(nt - 1);
}

// Workgroup = 8 waves, one (layer, 16-column tile, 16-unit half) over the whole
// batch: G[16 h + u][c0 + r] = sum over samples of delta[s][16 h + u] a_prev[s][c0 + r]
// on the 16x16x4 matrix cores.  Wave w takes every 8th group of 4 samples; the
// waves' sums are added in wave order, then the tile applies the SGD step.

constexpr int N2_WAVES = 8;
constexpr int N2_UNROLL = 32;  // groups of 4 samples loaded before use
constexpr int N2_RUN_ALIGN = 4;  // tiles per XCD run: a multiple of two column tiles x two halves

__global__ void __launch_bounds__(N2_WAVES * 64) narrow_dw_kernel(const NarrowDwParams p) {
  __shared__ float red[N2_WAVES][16][17];
  __shared__ float bred[N2_WAVES][4][16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // consecutive workgroups land on different XCDs (round robin over 8); the
  // grid is 8 runs of N2_RUN_ALIGN-aligned length, and XCD x takes the run of
  // tiles [x * per, (x + 1) * per), so the four tiles of two neighbouring
  // column tiles (both unit halves), whose 64-byte input slices share 128-byte
  // lines, meet in one L2; the grid's padding workgroups have no tile
  const int per = (int)gridDim.x >> 3;
  const int xcd = (int)blockIdx.x & 7, slot = (int)blockIdx.x >> 3;
  const int tile = xcd * per + slot;
  if (tile >= p.ntiles) return;
  // the layer of this tile (tile_base of the layers past the last is ntiles);
  // every per-layer argument is picked by value from constant indices, so
  // the argument loads all issue at kernel start
  const int l = (tile >= p.tile_base[1]) + (tile >= p.tile_base[2]) + (tile >= p.tile_base[3]);
  const int M = pick(l, p.dims[1], p.dims[2], p.dims[3], p.dims[4]);
  const int N = pick(l, p.dims[0], p.dims[1], p.dims[2], p.dims[3]);
  const int base = pick(l, p.tile_base[0], p.tile_base[1], p.tile_base[2], p.tile_base[3]);
  const int nh = (M + 15) / 16;
  const int c = (tile - base) / nh, h = (tile - base) % nh;
  const int c0 = c * 16, u0 = h * 16;
  const float* xop = pick(l, p.X, p.A[0], p.A[1], p.A[2]);
  const int64_t ldx = l == 0 ? p.dims[0] : NARROW_WIDTH;
  const float* dl = pick(l, p.D[0], p.D[1], p.D[2], p.D[3]) + u0;
  const int64_t ldw = pick(l, p.ldw[0], p.ldw[1], p.ldw[2], p.ldw[3]);
  float* G = pick(l, p.G[0], p.G[1], p.G[2], p.G[3]);
  float* W = pick(l, p.W[0], p.W[1], p.W[2], p.W[3]);
  const float* Win = pick(l, p.Win[0], p.Win[1], p.Win[2], p.Win[3]);
  float* gb = pick(l, p.gb[0], p.gb[1], p.gb[2], p.gb[3]);
  float* bias = pick(l, p.bias[0], p.bias[1], p.bias[2], p.bias[3]);
  const float* bin = pick(l, p.bin[0], p.bin[1], p.bin[2], p.bin[3]);

  // the parameters this thread updates at the end, requested now so that
  // their latency hides behind the batch loop (clamped, always valid)
  const int ui = (tid >> 4) & 15, uj = tid & 15;   // unit within the half, column within the tile
  const bool w_mine = tid < 256 && u0 + ui < M && c0 + uj < N;
  const int64_t wo = w_mine ? (int64_t)(u0 + ui) * ldw + c0 + uj : 0;
  const float w_old = Win[wo];
  const bool b_mine = c == 0 && tid < 16 && u0 + tid < M;
  const float b_old = bin[b_mine ? u0 + tid : 0];

  const int r = lane & 15, g = lane >> 4;
  const bool col_ok = c0 + r < N;
  const float* xcol = xop + (col_ok ? c0 + r : 0);
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  float bsum = 0.0f;
  const int ngroups = (p.B + 3) / 4;
  for (int g0 = wave; g0 < ngroups; g0 += N2_WAVES * N2_UNROLL) {
    float dv[N2_UNROLL], xv[N2_UNROLL];
#pragma unroll
    for (int u = 0; u < N2_UNROLL; ++u) {
      const int smp = (g0 + u * N2_WAVES) * 4 + g;
      const int sc = smp < p.B ? smp : p.B - 1;
      dv[u] = dl[(int64_t)sc * NARROW_WIDTH + r];
      xv[u] = xcol[(int64_t)sc * ldx];
    }
#pragma unroll
    for (int u = 0; u < N2_UNROLL; ++u) {
      const bool ok = (g0 + u * N2_WAVES) * 4 + g < p.B;
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

  float wn = 0.0f;
  if (w_mine) {
    float gsum = red[0][ui][uj];
#pragma unroll
    for (int w = 1; w < N2_WAVES; ++w) gsum += red[w][ui][uj];
    G[wo] = gsum;
    wn = fmaf(-p.scale, gsum, w_old);
    W[wo] = wn;
  }
  // layer 1: the tile's 16 x 16 block of the updated W_1 (zeros past d_1 and
  // d_0) into both packed copies; it is one whole block of W1i and a quarter
  // of four blocks of W1f
  if (l == 0 && tid < 256 && p.W1f) {
    const int u = u0 + ui, k = c0 + uj;
    p.W1i[((2 * c + h) * 64 + ui + 16 * (uj >> 2)) * 4 + (uj & 3)] = wn;
    p.W1f[(((k >> 6) * 8 + (u >> 2)) * 64 + 4 * ((k & 63) >> 2) + (u & 3)) * 4 + (k & 3)] = wn;
  }
  if (b_mine) {
    float gsum = 0.0f;
#pragma unroll
    for (int w = 0; w < N2_WAVES; ++w)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        gsum = (w == 0 && q == 0) ? bred[0][0][tid] : gsum + bred[w][q][tid];
    gb[u0 + tid] = gsum;
    bias[u0 + tid] = fmaf(-p.scale, gsum, b_old);
  }
}

// Both packed copies of W_1, one thread per packed element.
__global__ void __launch_bounds__(256) narrow_pack_w1_kernel(const float* W1, int64_t ldw, int d1,
                                                              int d0, float* W1f, float* W1i,
                                                              int64_t nf, int64_t ni) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < nf) {
    // W1f: block (t, q) = e / 256, lane 4 b + i, component v
    const int64_t blk = e >> 8;
    const int ln = (int)(e >> 2) & 63, v = (int)e & 3;
    const int t = (int)(blk >> 3), q = (int)blk & 7;
    const int u = 4 * q + (ln & 3), k = 64 * t + 4 * (ln >> 2) + v;
    W1f[e] = (u < d1 && k < d0) ? W1[(int64_t)u * ldw + k] : 0.0f;
  } else if (e < nf + ni) {
    // W1i: block (c, h) = (e - nf) / 256, lane r + 16 g, component v
    const int64_t f = e - nf;
    const int64_t blk = f >> 8;
    const int ln = (int)(f >> 2) & 63, v = (int)f & 3;
    const int c = (int)(blk >> 1), h = (int)blk & 1;
    const int u = 16 * h + (ln & 15), k = 16 * c + 4 * (ln >> 4) + v;
    W1i[f] = (u < d1 && k < d0) ? W1[(int64_t)u * ldw + k] : 0.0f;
  }
}

hipError_t launch_narrow_pack_w1(const float* W1, int64_t ldw, int d1, int d0, float* W1f,
                                 float* W1i, hipStream_t s) {
  const int64_t nf = narrow_pack_w1f_elems(d0), ni = narrow_pack_w1i_elems(d0);
  const dim3 grid((unsigned)((nf + ni + 255) / 256)), block(256);
  return launch_k(narrow_pack_w1_kernel, grid, block, 0, s, W1, ldw, d1, d0, W1f, W1i, nf, ni);
}

// The per-sample kernel for this pass: inference over batches above
// NARROW_SMALL_BATCH takes the persistent kernel when W_1 fits its matrix
// waves' registers (d0 <= 8 waves x NI_MC_MAX chunks x 16 = 1024) and every
// workgroup's input rows fit below NI_OOB bytes.
constexpr int NI_MC_MAX = 8;

int narrow_infer_grid(const NarrowFwdParams& p) {
  const int ntiles = (p.B + NARROW_TILE - 1) / NARROW_TILE;
  return ntiles < p.ncu ? ntiles : p.ncu;
}

NarrowKernel narrow_fwd_kernel(bool train, const NarrowFwdParams& p) {
  if (p.B <= NARROW_SMALL_BATCH) return NK_FWD4;
  if (!train && p.ncu > 0 && p.d0 <= NI_MW * NI_MC_MAX * NI_CH) {
    const int64_t ntiles = (p.B + NARROW_TILE - 1) / NARROW_TILE;
    const int64_t grid = narrow_infer_grid(p);
    const int64_t rows = (ntiles + grid - 1) / grid * NARROW_TILE;
    if (rows * p.d0 * 4 < (int64_t)NI_OOB) return NK_INFER;
  }
  return NK_FWD16;
}

hipError_t launch_narrow_fwd(bool train, const NarrowFwdParams& p, hipStream_t s) {
  const dim3 block(N1_WAVES * 64);
  switch (narrow_fwd_kernel(train, p)) {
    case NK_FWD4: {
      const dim3 grid((p.B + N4_T - 1) / N4_T);
      if (train)
        return launch_k(narrow_fwd4_kernel<true>, grid, block, 0, s, p);
      else
        return launch_k(narrow_fwd4_kernel<false>, grid, block, 0, s, p);
    }
    case NK_FWD16: {
      const dim3 grid((p.B + NARROW_TILE - 1) / NARROW_TILE);
      if (train)
        return launch_k(narrow_fwd16_kernel<true, N1_PRE_TRAIN>, grid, block, 0, s, p);
      else
        return launch_k(narrow_fwd16_kernel<false, N1_PRE_INFER>, grid, block, 0, s, p);
    }
    case NK_INFER: {
      const dim3 grid(narrow_infer_grid(p));
      // chunks per matrix wave
      switch (((p.d0 + NI_CH - 1) / NI_CH + NI_MW - 1) / NI_MW) {
        case 1: return launch_k(narrow_infer_kernel<1>, grid, block, 0, s, p);
        case 2: return launch_k(narrow_infer_kernel<2>, grid, block, 0, s, p);
        case 3: return launch_k(narrow_infer_kernel<3>, grid, block, 0, s, p);
        case 4: return launch_k(narrow_infer_kernel<4>, grid, block, 0, s, p);
        case 5: return launch_k(narrow_infer_kernel<5>, grid, block, 0, s, p);
        case 6: return launch_k(narrow_infer_kernel<6>, grid, block, 0, s, p);
        case 7: return launch_k(narrow_infer_kernel<7>, grid, block, 0, s, p);
        default: return launch_k(narrow_infer_kernel<NI_MC_MAX>, grid, block, 0, s, p);
      }
    }
  }
  return hipErrorInvalidValue;
}

const char* narrow_fwd_name(bool train, const NarrowFwdParams& p) {
  switch (narrow_fwd_kernel(train, p)) {
    case NK_FWD4:
      return train ? "narrow_fwd4_train" : "narrow_fwd4_infer";
    case NK_FWD16:
      return train ? "narrow_fwd16_train" : "narrow_fwd16_infer";
    default:
      return "narrow_infer";
  }
}

hipError_t launch_narrow_dw(const NarrowDwParams& p, hipStream_t s) {
  if (p.ntiles <= 0) return hipErrorInvalidValue;
  const int per = ((p.ntiles + 7) / 8 + N2_RUN_ALIGN - 1) / N2_RUN_ALIGN * N2_RUN_ALIGN;
  return launch_k(narrow_dw_kernel, dim3(8 * per), N2_WAVES * 64, 0, s, p);
}

}  // namespace nf
