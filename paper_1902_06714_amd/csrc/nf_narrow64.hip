// Training step and inference for narrow fp64 networks (the paper's real64
// kind, section 2; every layer after the input has at most 32 units), on the
// fp64 matrix cores.  Two kernels per step, as in fp32:
//   per-sample pass   one workgroup of 8 waves per 4-sample tile (batches up
//                     to NARROW_SMALL_BATCH, v_mfma_f64_4x4x4f64) or 16-sample
//                     tile (v_mfma_f64_16x16x4f64): layer 1 with the input
//                     width split over the waves and their sums added in a
//                     fixed order; layers 2..L, the output delta
//                     (a_L - y) f'(z_L) and the hidden deltas
//                     (W_{l+1}^T delta_{l+1}) f'(z_l) (section 3.3) one thread
//                     per (sample, unit) with the small layers in LDS;
//   tendencies + SGD  one workgroup per (layer, 16-column tile, 16-unit half)
//                     forms the batch sum of delta (outer) activation for its
//                     block, its waves splitting the batch and their sums
//                     added in wave order, and writes W' = W - (eta/B) G into
//                     the other parameter buffer (sections 3.3-3.5).
// The 16x16x4 fp64 instruction takes lane l's A entry (row l % 16, input
// l / 16) and B entry (input l / 16, column l % 16); accumulator register v of
// lane l holds row 4 v + l / 16, column l % 16.
// Every sum runs in a fixed order, so results are reproducible bit for bit.
#include "nf_act.h"
#include "nf_internal.h"

namespace nf {

typedef double doublex4 __attribute__((ext_vector_type(4)));

namespace {

// v if c, else zeros, per component
__device__ __forceinline__ double2 keep_if2(bool c, double2 v) {
  return make_double2(c ? v.x : 0.0, c ? v.y : 0.0);
}

constexpr int D_WAVES = 8;
constexpr int D_T = 16;                  // samples per tile
constexpr int D_CH = 8;                  // inputs per chunk: a 16-byte pair per lane group
constexpr int D_PRE = 4;                 // chunks per wave requested together
constexpr int D_NWP = NARROW_WIDTH + 2;  // LDS row pitch (16-byte aligned rows)
constexpr int D_NSTAGE = NARROW_WIDTH * NARROW_WIDTH / (D_WAVES * 64);
// an offset past every range read through a buffer resource: zeros, no access
constexpr unsigned D_OOB = NARROW_OOB;

// sum over i < 32 of w[i] h[i] from two 16-byte aligned LDS rows, in four
// interleaved partial sums added pairwise
__device__ __forceinline__ double dot32d(const double* w, const double* h) {
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int m = 0; m < NARROW_WIDTH / 4; ++m) {
    const double2 a0 = *reinterpret_cast<const double2*>(w + 4 * m);
    const double2 a1 = *reinterpret_cast<const double2*>(w + 4 * m + 2);
    const double2 x0 = *reinterpret_cast<const double2*>(h + 4 * m);
    const double2 x1 = *reinterpret_cast<const double2*>(h + 4 * m + 2);
    acc[0] = fma(a0.x, x0.x, acc[0]);
    acc[1] = fma(a0.y, x0.y, acc[1]);
    acc[2] = fma(a1.x, x1.x, acc[2]);
    acc[3] = fma(a1.y, x1.y, acc[3]);
  }
  return (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

// The weights of layers 2..L (padded 32 x 32 blocks, a zero block past the
// last layer) for LDS, and every layer's bias of unit tid % 32 (the unit the
// thread takes in the tail).  Loaded before layer 1, stored to LDS after it,
// so the loads land while layer 1 runs.
struct Small64 {
  double w[NARROW_MAX_LAYERS - 1][D_NSTAGE];
  double b[NARROW_MAX_LAYERS];
};

__device__ __forceinline__ void load_small64(const NarrowFwdParamsT<double>& p, int tid,
                                             Small64& r) {
#pragma unroll
  for (int li = 0; li < NARROW_MAX_LAYERS - 1; ++li)
#pragma unroll
    for (int u = 0; u < D_NSTAGE; ++u) r.w[li][u] = p.W[li + 1][tid + u * D_WAVES * 64];
#pragma unroll
  for (int l = 0; l < NARROW_MAX_LAYERS; ++l) r.b[l] = p.bias[l][tid & (NARROW_WIDTH - 1)];
}

// ws[l][j][i] = W(j, i) for the forward sums and, when training,
// wsT[l][i][j] = W(j, i) for the delta sums
template <bool TRANSPOSED>
__device__ __forceinline__ void store_small64(const Small64& r, int tid,
                                              double (*ws)[NARROW_WIDTH][D_NWP],
                                              double (*wsT)[NARROW_WIDTH][D_NWP]) {
  constexpr int NW = NARROW_WIDTH;
#pragma unroll
  for (int li = 0; li < NARROW_MAX_LAYERS - 1; ++li)
#pragma unroll
    for (int u = 0; u < D_NSTAGE; ++u) {
      const int e = tid + u * D_WAVES * 64;
      ws[li][e / NW][e % NW] = r.w[li][u];
      if (TRANSPOSED) wsT[li][e % NW][e / NW] = r.w[li][u];
    }
}

// target of (sample tid / 32, unit tid % 32) of a T-sample tile, read from a
// clamped position so the load carries no branch
template <int T>
__device__ __forceinline__ double load_target64(const NarrowFwdParamsT<double>& p, int s0,
                                                int tid) {
  const int ys = s0 + (tid >> 5), yu = tid & 31;
  const bool ok = tid < T * NARROW_WIDTH && ys < p.B && yu < p.dout;
  const int yr = ys < p.B ? ys : p.B - 1, yc = yu < p.dout ? yu : p.dout - 1;
  const double v = p.Y[(int64_t)yr * p.dout + yc];
  return ok ? v : 0.0;
}

// The tail's thread (s, j) = (tid / 32, tid % 32) keeps each sample's 32 units
// in one wave, so every phase of the tail reads only what its own wave wrote
// in the phase before: LDS operations of a wave complete in order, and a
// wavefront-scope fence keeps the compiler from moving them across the
// boundary.
__device__ __forceinline__ void tail_sync64() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Everything after the layer-1 sums, for thread (s, j) = (tid / 32, tid % 32):
// sample s of the T-sample tile, unit j.  Layer 1's activation, layers 2..L
// with the previous layer in LDS (padded units carry zeros, so every sum runs
// over 32), the output delta (a_L - y) f'(z_L) and the hidden deltas
// (W_{l+1}^T delta_{l+1}) f'(z_l) (section 3.3) with f'(z_l) kept in
// registers.  Threads past 32 T have no part in it.
template <bool TRAIN, int T>
__device__ __forceinline__ void narrow64_tail(const NarrowFwdParamsT<double>& p, int s0, int tid,
                                              double z1, double ytg, double (*hs)[T][D_NWP],
                                              const double (*ws)[NARROW_WIDTH][D_NWP],
                                              const double (*wsT)[NARROW_WIDTH][D_NWP],
                                              const double (&bias)[NARROW_MAX_LAYERS]) {
  constexpr int NW = NARROW_WIDTH;
  const bool active = T * NW >= D_WAVES * 64 || tid < T * NW;
  const int s = active ? tid >> 5 : 0, j = tid & 31;
  const int gs = s0 + s;
  const bool s_ok = active && gs < p.B;
  double fp[NARROW_MAX_LAYERS];
#pragma unroll
  for (int l = 0; l < NARROW_MAX_LAYERS; ++l) fp[l] = 0.0;
  int cur = 0;
  if (active) {
    double a = 0.0, f = 0.0;
    if (j < p.dims[1]) act_eval(p.acts[0], z1 + bias[0], a, f);
    fp[0] = f;
    if (p.L == 1) {
      if (TRAIN) {
        const double d = (j < p.dims[1] && s_ok) ? (a - ytg) * f : 0.0;
        if (s_ok) p.D[0][(int64_t)gs * NW + j] = d;
      } else if (s_ok && j < p.dims[1]) {
        p.out[(int64_t)gs * p.dims[1] + j] = a;
      }
    } else {
      hs[0][s][j] = a;
      if (TRAIN && s_ok) p.A[0][(int64_t)gs * NW + j] = a;
    }
  }
  tail_sync64();

  // ---- layers 2..L
#pragma unroll
  for (int l = 2; l <= NARROW_MAX_LAYERS; ++l) {
    if (l > p.L) break;
    if (active) {
      const int dl = p.dims[l];
      const double z = dot32d(ws[l - 2][j], hs[cur][s]);
      double a = 0.0, f = 0.0;
      if (j < dl) act_eval(p.acts[l - 1], z + bias[l - 1], a, f);
      fp[l - 1] = f;
      if (l == p.L) {
        if (TRAIN) {
          const double d = (j < dl && s_ok) ? (a - ytg) * f : 0.0;
          hs[cur ^ 1][s][j] = d;
          if (s_ok) p.D[l - 1][(int64_t)gs * NW + j] = d;
        } else if (s_ok && j < dl) {
          p.out[(int64_t)gs * dl + j] = a;
        }
      } else {
        hs[cur ^ 1][s][j] = a;
        if (TRAIN && s_ok) p.A[l - 1][(int64_t)gs * NW + j] = a;
      }
    }
    cur ^= 1;
    tail_sync64();
  }
  if (!TRAIN) return;

  // ---- hidden deltas, l = L-1 .. 1, with the weights W_{l+1} of this step
  // (layer 1's delta is read by no later phase: no LDS copy, no barrier)
#pragma unroll
  for (int l = NARROW_MAX_LAYERS - 1; l >= 1; --l) {
    if (l >= p.L) continue;
    if (active) {
      const double t = dot32d(wsT[l - 1][j], hs[cur][s]);
      const double d = j < p.dims[l] ? t * fp[l - 1] : 0.0;
      if (l > 1) hs[cur ^ 1][s][j] = d;
      if (s_ok) p.D[l - 1][(int64_t)gs * NW + j] = d;
    }
    cur ^= 1;
    if (l > 1) tail_sync64();
  }
}

// 4-sample tiles: layer 1 on v_mfma_f64_4x4x4f64, whose four 4x4x4 blocks
// take lane l = 16 k + 4 b + x as row x, input k of block b's A and input k,
// column x of its B, and leave block b's (i, j) entry in lane 16 i + 4 b + j.
constexpr int D4_T = 4;                    // samples per tile
constexpr int D4_KS = 32;                  // inputs per step: one 16-byte pair per (block, input) lane
constexpr int D4_PRE = 4;                  // steps per wave requested together
constexpr int D4_UG = NARROW_WIDTH / 4;    // groups of 4 units
constexpr int D4_PARTS = D_WAVES * 4;      // (wave, block) sums of each output
constexpr int D4_RP = NARROW_WIDTH + 4;    // row pitch of the sums: a wave's 16-lane groups write 32 banks
constexpr int D4_SS = D4_PARTS * D4_RP;    // sample stride of the sums

}  // namespace

template <bool TRAIN>
__global__ void __launch_bounds__(D_WAVES * 64) narrow64_fwd_kernel(const NarrowFwdParamsT<double> p) {
  constexpr int T = D_T;
  constexpr int NW = NARROW_WIDTH;
  __shared__ double zp[D_WAVES][T][NW + 1];                         // the waves' layer-1 sums
  __shared__ __attribute__((aligned(16))) double hs[2][T][D_NWP];   // activations, then deltas
  __shared__ __attribute__((aligned(16))) double ws[NARROW_MAX_LAYERS - 1][NW][D_NWP];
  __shared__ __attribute__((aligned(16))) double wsT[TRAIN ? NARROW_MAX_LAYERS - 1 : 1][NW][D_NWP];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int s0 = blockIdx.x * T;

  Small64 sl;
  load_small64(p, tid, sl);
  const double ytg = TRAIN ? load_target64<T>(p, s0, tid) : 0.0;

  // ---- layer 1: lane (r, g) = (lane % 16, lane / 16) feeds sample r and
  // units r, 16 + r with inputs 8 c + 2 g and 8 c + 2 g + 1 of chunk c (one
  // per instruction); wave w takes chunks w, w + 8, ...  W_1 rows are padded
  // to 32 with zeros; the input width is even, so a pair is wholly in or out.
  {
    const int r = lane & 15, g = lane >> 4;
    const int nch = (p.d0 + D_CH - 1) / D_CH;
    const bool xrow_ok = s0 + r < p.B;
    const double* xsrc = p.X + (int64_t)(xrow_ok ? s0 + r : p.B - 1) * p.d0;
    const double* wsrc0 = p.W[0] + (int64_t)r * p.ldw[0];
    const double* wsrc1 = p.W[0] + (int64_t)(16 + r) * p.ldw[0];
    doublex4 acc0 = {0.0, 0.0, 0.0, 0.0}, acc1 = {0.0, 0.0, 0.0, 0.0};
    for (int c0 = wave; c0 < nch; c0 += D_WAVES * D_PRE) {
      double2 xr[D_PRE], w0[D_PRE], w1[D_PRE];
#pragma unroll
      for (int u = 0; u < D_PRE; ++u) {
        const int k = (c0 + D_WAVES * u) * D_CH + 2 * g;
        const bool ok = k < p.d0;
        const int kc = ok ? k : 0;
        xr[u] = keep_if2(ok && xrow_ok, *reinterpret_cast<const double2*>(xsrc + kc));
        w0[u] = keep_if2(ok, *reinterpret_cast<const double2*>(wsrc0 + kc));
        w1[u] = keep_if2(ok, *reinterpret_cast<const double2*>(wsrc1 + kc));
      }
#pragma unroll
      for (int u = 0; u < D_PRE; ++u) {
        acc0 = __builtin_amdgcn_mfma_f64_16x16x4f64(xr[u].x, w0[u].x, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f64_16x16x4f64(xr[u].x, w1[u].x, acc1, 0, 0, 0);
        acc0 = __builtin_amdgcn_mfma_f64_16x16x4f64(xr[u].y, w0[u].y, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f64_16x16x4f64(xr[u].y, w1[u].y, acc1, 0, 0, 0);
      }
    }
    // accumulator register v of lane (r, g): sample 4 v + g, unit r (+16)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      zp[wave][4 * v + g][r] = acc0[v];
      zp[wave][4 * v + g][16 + r] = acc1[v];
    }
  }
  store_small64<TRAIN>(sl, tid, ws, wsT);
  __syncthreads();

  // the waves' sums in wave order
  double z1 = 0.0;
  {
    const int s = tid >> 5, j = tid & 31;
    z1 = zp[0][s][j];
#pragma unroll
    for (int w = 1; w < D_WAVES; ++w) z1 += zp[w][s][j];
  }
  narrow64_tail<TRAIN, T>(p, s0, tid, z1, ytg, hs, ws, wsT, sl.b);
}

// One workgroup of 8 waves per 4-sample tile (batches up to
// NARROW_SMALL_BATCH, so a 1000-sample batch spreads over 250 CUs).  Layer 1:
// lane (k, b, x) = (lane / 16, lane / 4 % 4, lane % 4) loads a 16-byte pair of
// sample x's row and of W_1 rows 4 g + x (the 8 unit groups g) at inputs
// 32 t + 2 (4 b + k) and + 1 of step t; the pair's two elements feed two
// instructions per unit group.  Block b of wave w thus sums its own inputs,
// and the 32 (wave, block) sums of each output are added in a fixed order.
template <bool TRAIN>
__global__ void __launch_bounds__(D_WAVES * 64) narrow64_fwd4_kernel(const NarrowFwdParamsT<double> p) {
  constexpr int T = D4_T;
  constexpr int NW = NARROW_WIDTH;
  __shared__ double red[T * D4_SS];                                 // [sample][wave*4+block][unit]
  __shared__ double psum[4][T][NW];
  __shared__ __attribute__((aligned(16))) double hs[2][T][D_NWP];
  __shared__ __attribute__((aligned(16))) double ws[NARROW_MAX_LAYERS - 1][NW][D_NWP];
  __shared__ __attribute__((aligned(16))) double wsT[TRAIN ? NARROW_MAX_LAYERS - 1 : 1][NW][D_NWP];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int s0 = blockIdx.x * T;

  Small64 sl;
  load_small64(p, tid, sl);
  const double ytg = TRAIN ? load_target64<T>(p, s0, tid) : 0.0;

  {
    const int x = lane & 3, b = (lane >> 2) & 3, kq = lane >> 4;
    const int pos = 4 * b + kq;
    // the tile's input rows and W_1's d_1 rows through buffer resources that
    // end at the last row: rows past the batch, W_1's padding rows and inputs
    // past the width (given an offset past the end) read as zeros without a
    // memory access.  The width is even, so a pair is wholly in or out.
    const int nrows = p.B - s0 < T ? p.B - s0 : T;
    const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(p.X + (int64_t)s0 * p.d0), (short)0, nrows * p.d0 * 8, 0x00020000);
    const int ldw1 = (int)p.ldw[0];
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        (void*)p.W[0], (short)0, p.dims[1] * ldw1 * 8, 0x00020000);
    double acc[D4_UG];
#pragma unroll
    for (int ug = 0; ug < D4_UG; ++ug) acc[ug] = 0.0;
    const int nsteps = (p.d0 + D4_KS - 1) / D4_KS;
    // workgroups start at different steps (rotated by the tile index), so the
    // workgroups that start together do not all ask for the same W_1 lines
    const int rot = (int)(blockIdx.x % (unsigned)nsteps);
    // the first block of steps runs unconditionally (a wave without steps adds
    // zeros), so its loads are not held behind a branch
    int t0 = wave;
    do {
      double2 xr[D4_PRE], wr[D4_PRE][D4_UG];
#pragma unroll
      for (int u = 0; u < D4_PRE; ++u) {
        int t = t0 + u * D_WAVES;
        if (t < nsteps) t = t + rot < nsteps ? t + rot : t + rot - nsteps;
        const int k = t * D4_KS + 2 * pos;
        const bool ok = k < p.d0;
        xr[u] = __builtin_bit_cast(double2, __builtin_amdgcn_raw_buffer_load_b128(
                                                xres, ok ? 8 * (x * p.d0 + k) : (int)D_OOB, 0, 0));
#pragma unroll
        for (int ug = 0; ug < D4_UG; ++ug)
          wr[u][ug] = __builtin_bit_cast(
              double2, __builtin_amdgcn_raw_buffer_load_b128(
                           wres, ok ? 8 * ((4 * ug + x) * ldw1 + k) : (int)D_OOB, 0, 0));
      }
      // keep every load of the block ahead of the first matrix instruction
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < D4_PRE; ++u) {
#pragma unroll
        for (int ug = 0; ug < D4_UG; ++ug)
          acc[ug] = __builtin_amdgcn_mfma_f64_4x4x4f64(xr[u].x, wr[u][ug].x, acc[ug], 0, 0, 0);
#pragma unroll
        for (int ug = 0; ug < D4_UG; ++ug)
          acc[ug] = __builtin_amdgcn_mfma_f64_4x4x4f64(xr[u].y, wr[u][ug].y, acc[ug], 0, 0, 0);
      }
      t0 += D_WAVES * D4_PRE;
    } while (t0 < nsteps);
    // lane (i, b, j) = (lane / 16, lane / 4 % 4, lane % 4) holds block b's sum
    // for sample i, unit 4 g + j
    const int i = lane >> 4, j = lane & 3;
#pragma unroll
    for (int ug = 0; ug < D4_UG; ++ug)
      red[i * D4_SS + (wave * 4 + b) * D4_RP + 4 * ug + j] = acc[ug];
  }
  store_small64<TRAIN>(sl, tid, ws, wsT);
  __syncthreads();

  // every thread adds a quarter of the (wave, block) sums of one output, in
  // order; the quarters are then added pairwise
  {
    const int part = tid >> 7, s = (tid >> 5) & 3, j = tid & 31;
    const double* src = red + s * D4_SS + part * (D4_PARTS / 4) * D4_RP + j;
    double t = src[0];
#pragma unroll
    for (int r = 1; r < D4_PARTS / 4; ++r) t += src[r * D4_RP];
    psum[part][s][j] = t;
  }
  __syncthreads();
  double z1 = 0.0;
  if (tid < T * NW) {
    const int s = tid >> 5, j = tid & 31;
    z1 = (psum[0][s][j] + psum[1][s][j]) + (psum[2][s][j] + psum[3][s][j]);
  }
  narrow64_tail<TRAIN, T>(p, s0, tid, z1, ytg, hs, ws, wsT, sl.b);
}

// Workgroup = 8 waves, one (layer, 16-column tile, 16-unit half) over the
// whole batch: G[16 h + u][c0 + r] = sum over samples of
// delta[s][16 h + u] a_prev[s][c0 + r].  Wave w takes every 8th group of 4
// samples; the waves' sums are added in wave order, then the tile applies the
// SGD step.
namespace {

template <class V>
__device__ __forceinline__ V pick4(int l, V a0, V a1, V a2, V a3) {
  return l == 0 ? a0 : (l == 1 ? a1 : (l == 2 ? a2 : a3));
}

constexpr int D2_WAVES = 8;
constexpr int D2_UNROLL = 16;  // groups of 4 samples loaded before use

}  // namespace

__global__ void __launch_bounds__(D2_WAVES * 64) narrow64_dw_kernel(const NarrowDwParamsT<double> p) {
  __shared__ double red[D2_WAVES][16][17];
  __shared__ double bred[D2_WAVES][4][16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // consecutive workgroups land on different XCDs (round robin over 8); give
  // each XCD a contiguous run of tiles, so the two unit halves of a column
  // tile and neighbouring column tiles share the input rows in one L2
  const int nwg = p.ntiles;
  const int per = (nwg + 7) / 8;
  const int full = nwg - 8 * (per - 1);
  const int xcd = (int)blockIdx.x & 7, slot = (int)blockIdx.x >> 3;
  const int tile = xcd < full ? xcd * per + slot : full * per + (xcd - full) * (per - 1) + slot;
  const int l = (tile >= p.tile_base[1]) + (tile >= p.tile_base[2]) + (tile >= p.tile_base[3]);
  const int M = pick4(l, p.dims[1], p.dims[2], p.dims[3], p.dims[4]);
  const int N = pick4(l, p.dims[0], p.dims[1], p.dims[2], p.dims[3]);
  const int base = pick4(l, p.tile_base[0], p.tile_base[1], p.tile_base[2], p.tile_base[3]);
  const int nh = (M + 15) / 16;
  const int c = (tile - base) / nh, h = (tile - base) % nh;
  const int c0 = c * 16, u0 = h * 16;
  const double* xop = pick4(l, p.X, p.A[0], p.A[1], p.A[2]);
  const int64_t ldx = l == 0 ? p.dims[0] : NARROW_WIDTH;
  const double* dl = pick4(l, p.D[0], p.D[1], p.D[2], p.D[3]) + u0;
  const int64_t ldw = pick4(l, p.ldw[0], p.ldw[1], p.ldw[2], p.ldw[3]);
  double* G = pick4(l, p.G[0], p.G[1], p.G[2], p.G[3]);
  double* W = pick4(l, p.W[0], p.W[1], p.W[2], p.W[3]);
  const double* Win = pick4(l, p.Win[0], p.Win[1], p.Win[2], p.Win[3]);
  double* gb = pick4(l, p.gb[0], p.gb[1], p.gb[2], p.gb[3]);
  double* bias = pick4(l, p.bias[0], p.bias[1], p.bias[2], p.bias[3]);
  const double* bin = pick4(l, p.bin[0], p.bin[1], p.bin[2], p.bin[3]);

  // the parameters this thread updates at the end, requested now (clamped,
  // always valid)
  const int ui = (tid >> 4) & 15, uj = tid & 15;
  const bool w_mine = tid < 256 && u0 + ui < M && c0 + uj < N;
  const int64_t wo = w_mine ? (int64_t)(u0 + ui) * ldw + c0 + uj : 0;
  const double w_old = Win[wo];
  const bool b_mine = c == 0 && tid < 16 && u0 + tid < M;
  const double b_old = bin[b_mine ? u0 + tid : 0];

  // lane (r, g) feeds unit u0 + r and column c0 + r with sample g of each
  // group of 4 (one instruction per group)
  const int r = lane & 15, g = lane >> 4;
  const bool col_ok = c0 + r < N;
  const double* xcol = xop + (col_ok ? c0 + r : 0);
  doublex4 acc = {0.0, 0.0, 0.0, 0.0};
  double bsum = 0.0;
  const int ngroups = (p.B + 3) / 4;
  for (int g0 = wave; g0 < ngroups; g0 += D2_WAVES * D2_UNROLL) {
    double dv[D2_UNROLL], xv[D2_UNROLL];
#pragma unroll
    for (int u = 0; u < D2_UNROLL; ++u) {
      const int smp = (g0 + u * D2_WAVES) * 4 + g;
      const int sc = smp < p.B ? smp : p.B - 1;
      dv[u] = dl[(int64_t)sc * NARROW_WIDTH + r];
      xv[u] = xcol[(int64_t)sc * ldx];
    }
#pragma unroll
    for (int u = 0; u < D2_UNROLL; ++u) {
      const bool ok = (g0 + u * D2_WAVES) * 4 + g < p.B;
      const double a = ok ? dv[u] : 0.0;
      const double b = (ok && col_ok) ? xv[u] : 0.0;
      acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc, 0, 0, 0);
      bsum += a;
    }
  }
  // accumulator register v of lane (r, g): unit u0 + 4 v + g, column c0 + r
#pragma unroll
  for (int v = 0; v < 4; ++v) red[wave][4 * v + g][r] = acc[v];
  if (c == 0) bred[wave][g][r] = bsum;
  __syncthreads();

  if (w_mine) {
    double gsum = red[0][ui][uj];
#pragma unroll
    for (int w = 1; w < D2_WAVES; ++w) gsum += red[w][ui][uj];
    G[wo] = gsum;
    W[wo] = fma(-p.scale, gsum, w_old);
  }
  if (b_mine) {
    double gsum = 0.0;
#pragma unroll
    for (int w = 0; w < D2_WAVES; ++w)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        gsum = (w == 0 && q == 0) ? bred[0][0][tid] : gsum + bred[w][q][tid];
    gb[u0 + tid] = gsum;
    bias[u0 + tid] = fma(-p.scale, gsum, b_old);
  }
}

hipError_t launch_narrow64_fwd(bool train, const NarrowFwdParamsT<double>& p, hipStream_t s) {
  if (p.B <= NARROW_SMALL_BATCH) {
    const dim3 grid((p.B + D4_T - 1) / D4_T);
    if (train)
      return launch_k(narrow64_fwd4_kernel<true>, grid, D_WAVES * 64, 0, s, p);
    else
      return launch_k(narrow64_fwd4_kernel<false>, grid, D_WAVES * 64, 0, s, p);
  }
  const dim3 grid((p.B + D_T - 1) / D_T);
  if (train)
    return launch_k(narrow64_fwd_kernel<true>, grid, D_WAVES * 64, 0, s, p);
  else
    return launch_k(narrow64_fwd_kernel<false>, grid, D_WAVES * 64, 0, s, p);
}

const char* narrow64_fwd_name(bool train, const NarrowFwdParamsT<double>& p) {
  if (p.B <= NARROW_SMALL_BATCH) return train ? "narrow64_fwd4_train" : "narrow64_fwd4_infer";
  return train ? "narrow64_fwd_train" : "narrow64_fwd_infer";
}

hipError_t launch_narrow64_dw(const NarrowDwParamsT<double>& p, hipStream_t s) {
  return launch_k(narrow64_dw_kernel, dim3(p.ntiles), D2_WAVES * 64, 0, s, p);
}

}  // namespace nf
