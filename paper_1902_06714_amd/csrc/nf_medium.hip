// Per-sample pass for networks whose layers after the input have at most 128
// units (e.g. 784-100-100-10), in fp32 and fp64.  Layer 1's contraction runs before it
// (its k pieces in the piece buffer); then each workgroup of 12 waves, for
// tiles of 16 NSB samples,
//   folds layer 1's pieces in piece order, adds b_1 and applies f_1;
//   runs layers 2..L with the weights of layers 2..L staged in LDS;
//   forms the output delta (a_L - y) f'(z_L) and the hidden deltas
//   (W_{l+1}^T delta_{l+1}) f'(z_l) (section 3.3) with the weights of this
//   step;
// and stores the activations and deltas the tendency kernels read.  Every
// product is on the 16x16x4 matrix cores of the element type (fp32 or fp64;
// both take lane (r, g)'s inputs as row r / column r and input g, and differ
// in where accumulator register v lands: row 4 g + v in fp32, 4 v + g in
// fp64).  The work of a layer is split
// into jobs of 16 units x 16 samples, handed to the waves round robin; a
// layer's forward product and its delta use the same jobs, so the lane that
// formed f'(z_l) for a (sample, unit) forms that delta and keeps f' in
// registers.  Sums run in a fixed order, so results are reproducible bit for
// bit.
//
// Workgroups are persistent (one per CU): the weights are staged once, and
// the layer-1 pieces and targets of a workgroup's next tile are loaded while
// it works on the current one.  Per-sample loads and stores go through buffer
// resources, with lanes off the tile given an offset past the end, so every
// lane issues the same memory instructions and a wait for a prefetched value
// never waits for the stores issued after it.  A lane's offsets are 32-bit:
// its place in the tile in the vector offset, the tile's in the scalar one.
#include <type_traits>

#include "nf_act.h"
#include "nf_internal.h"

namespace nf {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef double doublex4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int M_WAVES = 12;
constexpr int M_THREADS = M_WAVES * 64;
// LDS row pitch of activations and deltas.  The matrix-core operand reads
// take 16 rows x 2 columns per half-wave; a pitch of 2 mod 32 (in 4-byte
// banks) puts them in 32 different banks.
constexpr int M_HP = MEDIUM_WIDTH + 2;
constexpr int M_PF = 2;                 // layer-1 pieces loaded ahead per tile
constexpr int M_STAGE = 8;              // weight loads in flight per thread

__device__ inline __amdgpu_buffer_rsrc_t rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)MEDIUM_OOB,
                                           0x00020000);
}
// the element type's matrix instruction, accumulator and layout
template <class T>
struct MedT;
template <>
struct MedT<float> {
  using acc_t = floatx4;
  using vec16 = float4;
  static constexpr int RS = 1, GS = 4;  // tile row of register v of lane group g: GS g + RS v
  static constexpr int WLDS = MEDIUM_LDS_WEIGHTS;
  __device__ static acc_t mma(float a, float b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  __device__ static float load(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
    return __builtin_bit_cast(float,
                              __builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, 0));
  }
  __device__ static void store(float v, __amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, (int)voff,
                                          (int)soff, 0);
  }
};
template <>
struct MedT<double> {
  using acc_t = doublex4;
  using vec16 = double2;
  static constexpr int RS = 4, GS = 1;
  static constexpr int WLDS = MEDIUM64_LDS_WEIGHTS;
  __device__ static acc_t mma(double a, double b, acc_t c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
  }
  __device__ static double load(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
    return __builtin_bit_cast(double,
                              __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, (int)soff, 0));
  }
  __device__ static void store(double v, __amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, v), r, (int)voff, (int)soff, 0);
  }
};

// calls f with the activation as a compile-time constant, so the code of one
// phase holds one activation's arithmetic, not a switch per element
template <class F>
__device__ __forceinline__ void with_act(int act, F&& f) {
  switch (act) {
    case ACT_SIGMOID: f(std::integral_constant<int, ACT_SIGMOID>{}); break;
    case ACT_TANH: f(std::integral_constant<int, ACT_TANH>{}); break;
    case ACT_RELU: f(std::integral_constant<int, ACT_RELU>{}); break;
    case ACT_GAUSSIAN: f(std::integral_constant<int, ACT_GAUSSIAN>{}); break;
    default: f(std::integral_constant<int, ACT_STEP>{}); break;
  }
}

}  // namespace

template <class T, int NSB, int L>
__global__ void __launch_bounds__(M_THREADS) medium_kernel(const MediumParamsT<T> p) {
  using M = MedT<T>;
  constexpr int TS = 16 * NSB;                       // samples per tile
  constexpr int NJ = (8 * NSB + M_WAVES - 1) / M_WAVES;  // jobs per wave at most
  constexpr unsigned SZ = sizeof(T);
  constexpr int VW = 16 / sizeof(T);                  // elements per 16-byte load
  constexpr int LPR = MEDIUM_WIDTH / VW;              // lanes per staged weight row
  constexpr int SROWS = M_THREADS / LPR;              // weight rows per load
  // one LDS block: the activations and deltas first, so that their reads
  // take immediate offsets, then W_2 .. W_L (padded), b_1 .. b_L and a spare
  // 16-byte slot
  constexpr int HSZ = 2 * TS * M_HP;
  __shared__ __attribute__((aligned(16))) T sm[HSZ + M::WLDS + L * MEDIUM_WIDTH + 16 / sizeof(T)];
  T(*const hs)[TS][M_HP] = reinterpret_cast<T(*)[TS][M_HP]>(sm);
  T* const wl = sm + HSZ;
  T(*const bl)[MEDIUM_WIDTH] = reinterpret_cast<T(*)[MEDIUM_WIDTH]>(sm + HSZ + M::WLDS);
  float4* const spare = reinterpret_cast<float4*>(sm + HSZ + M::WLDS + L * MEDIUM_WIDTH);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, g = lane >> 4;
  const int ntiles = (p.B + TS - 1) / TS;
  const int d1 = p.dims[1], dL = p.dims[L];
  const int ldz = (int)p.ldz;

  // job jj of this wave in a layer of d units: job = wave + 12 jj, unit block
  // job / NSB, sample block job % NSB; lane (r, g) holds unit 16 ub + r and,
  // in accumulator register v, tile row row(jj) + RS v (16 sb + 4 g + v in
  // fp32, 16 sb + g + 4 v in fp64)
  auto has_job = [&](int jj, int d) { return wave + M_WAVES * jj < ((d + 15) >> 4) * NSB; };
  auto unit = [&](int jj) { return 16 * ((wave + M_WAVES * jj) / NSB) + r; };
  auto sblk = [&](int jj) { return 16 * ((wave + M_WAVES * jj) % NSB); };
  auto row = [&](int jj) { return sblk(jj) + M::GS * g; };
  constexpr int RS = M::RS;

  const __amdgpu_buffer_rsrc_t zres = rsrc(p.zp), yres = rsrc(p.Y);

  // layer-1 pieces 0 .. M_PF-1 and the targets of tile tt (a tile past the
  // last loads nothing: every row is past the batch, and its scalar offsets
  // are the last tile's)
  T pz[M_PF][NJ][4], py[NJ][4];
  auto load_z = [&](int tt) {
    const int rem = p.B - tt * TS, tc = tt < ntiles ? tt : ntiles - 1;
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) {
      if (!has_job(jj, d1)) break;
      const int u = unit(jj), rw = row(jj);
      const unsigned vb = SZ * (unsigned)(rw * ldz + u);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const bool ok = u < d1 && rw + RS * v < rem;
#pragma unroll
        for (int q = 0; q < M_PF; ++q) {
          const int qq = q < p.np ? q : 0;
          pz[q][jj][v] = M::load(zres, ok ? vb : MEDIUM_OOB,
                                 SZ * (unsigned)((tc * TS + RS * v) * ldz + qq * (int)p.zstride));
        }
      }
    }
  };
  auto load_y = [&](int tt) {
    const int rem = p.B - tt * TS, tc = tt < ntiles ? tt : ntiles - 1;
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) {
      if (!has_job(jj, dL)) break;
      const int u = unit(jj), rw = row(jj);
      const unsigned vb = SZ * (unsigned)(rw * dL + u);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const bool ok = u < dL && rw + RS * v < rem;
        py[jj][v] = M::load(yres, ok ? vb : MEDIUM_OOB, SZ * (unsigned)((tc * TS + RS * v) * dL));
      }
    }
  };
  // b_1 of this lane's units, kept in registers for every tile
  T b1r[NJ];
#pragma unroll
  for (int jj = 0; jj < NJ; ++jj) {
    const int u = unit(jj);
    const bool ok = has_job(jj, d1) && u < d1;
    const T b = p.bias[0][ok ? u : 0];
    b1r[jj] = ok ? b : T(0);
  }

  // b_l for LDS, zero past d_l (128 threads, two whole waves, per layer).  The
  // load issues here, with the others; the value goes to LDS after the weight
  // loads have issued, so the prologue waits for memory once.
  const int bl_u = tid % MEDIUM_WIDTH;
  const bool bl_mine = tid < L * MEDIUM_WIDTH;
  // MEDIUM_WIDTH threads are whole waves: the layer is uniform in a wave, so
  // its size and bias pointer come from scalar loads
  const int bl_w = __builtin_amdgcn_readfirstlane(tid / MEDIUM_WIDTH) + 1;
  const int bl_l = bl_w < L ? bl_w : L;
  const bool bl_ok = bl_mine && bl_u < p.dims[bl_l];
  const T bl_v = p.bias[bl_l - 1][bl_ok ? bl_u : 0];

  T fp[L - 1][NJ][4];  // f'(z_l), l < L

  // ---- layer 1 of tile t: the pieces of z_1 in piece order, + b_1, f_1;
  // the next tile's pieces are requested once these are summed
  auto layer1 = [&](int t) {
    const int s0 = t * TS, rem = p.B - s0;
    T zs[NJ][4];
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        zs[jj][v] = pz[0][jj][v];
#pragma unroll
        for (int q = 1; q < M_PF; ++q)
          if (q < p.np) zs[jj][v] += pz[q][jj][v];
      }
    // pieces past those loaded ahead (small batches cut into many pieces)
    for (int q = M_PF; q < p.np; ++q) {
      T tq[NJ][4];
#pragma unroll
      for (int jj = 0; jj < NJ; ++jj) {
        if (!has_job(jj, d1)) break;
        const int u = unit(jj), rw = row(jj);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const bool ok = u < d1 && rw + RS * v < rem;
          tq[jj][v] = M::load(zres, ok ? SZ * (unsigned)(rw * ldz + u) : MEDIUM_OOB,
                              SZ * (unsigned)((s0 + RS * v) * ldz + q * (int)p.zstride));
        }
      }
#pragma unroll
      for (int jj = 0; jj < NJ; ++jj)
#pragma unroll
        for (int v = 0; v < 4; ++v) zs[jj][v] += tq[jj][v];
    }
    load_z(t + gridDim.x);
    const __amdgpu_buffer_rsrc_t ares = rsrc(p.A[0]);
    const int lda = (int)p.lda[0];
    with_act(p.acts[0], [&](auto act) {
#pragma unroll
      for (int jj = 0; jj < NJ; ++jj) {
        if (!has_job(jj, d1)) break;
        const int u = unit(jj), rw = row(jj);
        const unsigned vb = SZ * (unsigned)(rw * lda + u);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const bool ok = u < d1 && rw + RS * v < rem;
          T a, f;
          act_eval(decltype(act)::value, zs[jj][v] + b1r[jj], a, f);
          a = ok ? a : T(0);
          M::store(a, ares, ok ? vb : MEDIUM_OOB, SZ * (unsigned)((s0 + RS * v) * lda));
          hs[0][rw + RS * v][u] = a;
          fp[0][jj][v] = f;
        }
      }
    });
  };

  // the weights of layers 2..L into LDS: a row is 128 elements, 16 bytes a lane
  // (32 lanes in fp32, 64 in fp64).
  // Staged row R (over the layers' padded rows in order) is row j of layer l;
  // rows of the device layout are 16-byte aligned with a zero-filled pitch,
  // and rows past d_l and columns past that pitch are stored as zeros, so
  // every product below runs over whole 16-unit blocks (the bank padding at
  // the end of each LDS row is never read).  The LDS pitch is 18 mod 32
  // elements, so fp32 rows are 8-byte aligned: each 16-byte load is stored as
  // two 8-byte halves.  The first round of these loads (from the L2) issues
  // before the first tile's layer-1 pieces and targets (from memory): a CU
  // keeps a bounded number of loads in flight, so weight loads queued behind
  // them would arrive at their pace.  The weights are stored to LDS while the
  // pieces are on their way.
  {
    int rend[L];  // staged rows of layers 2..l
    rend[1] = p.wrows[1];
#pragma unroll
    for (int l = 3; l <= L; ++l) rend[l - 1] = rend[l - 2] + p.wrows[l - 1];
    const int rtot = rend[L - 1];
    const int c = VW * (tid % LPR);
    typename M::vec16 v[M_STAGE];
    int dst[M_STAGE];
    auto stage_issue = [&](int R0) {
#pragma unroll
      for (int i = 0; i < M_STAGE; ++i) {
        const int R = R0 + i * SROWS;
        int li = 1, r0 = 0;
#pragma unroll
        for (int l = 3; l <= L; ++l)
          if (R >= rend[l - 2]) li = l - 1, r0 = rend[l - 2];
        const int j = R - r0;
        // the layer's figures by selects (li differs between lanes)
        auto pick = [&](auto a1, auto a2, auto a3) { return li == 1 ? a1 : li == 2 ? a2 : a3; };
        const int wp = pick(p.wp[1], p.wp[2], p.wp[3]);
        const int cw = (pick(p.dims[1], p.dims[2], p.dims[3]) + 15) & ~15;  // padded width
        const int ldw = (int)pick(p.ldw[1], p.ldw[2], p.ldw[3]);
        const int dl = pick(p.dims[2], p.dims[3], p.dims[4]);
        const T* W = pick(p.W[1], p.W[2], p.W[3]);
        const bool in = R < rtot && c < cw;
        const bool ok = in && j < dl && c < ldw;
        const typename M::vec16 x =
            *reinterpret_cast<const typename M::vec16*>(ok ? W + (int64_t)j * ldw + c : p.W[1]);
        v[i] = ok ? x : typename M::vec16{};
        dst[i] = in ? pick(p.woff[1], p.woff[2], p.woff[3]) + j * wp + c : -1;
      }
    };
    // rows past the last layer and columns past the padded width go to a
    // spare slot, so no load is tied to a branch
    auto stage_store = [&]() {
#pragma unroll
      for (int i = 0; i < M_STAGE; ++i) {
        if constexpr (sizeof(T) == 4) {
          float2* d = dst[i] >= 0 ? reinterpret_cast<float2*>(wl + dst[i])
                                  : reinterpret_cast<float2*>(spare);
          d[0] = make_float2(v[i].x, v[i].y);
          d[1] = make_float2(v[i].z, v[i].w);
        } else {
          *(dst[i] >= 0 ? reinterpret_cast<double2*>(wl + dst[i])
                        : reinterpret_cast<double2*>(spare)) = v[i];
        }
      }
    };
    stage_issue(tid / LPR);
    load_z(blockIdx.x);  // the grid has at most one workgroup per tile
    load_y(blockIdx.x);
    stage_store();
    layer1(blockIdx.x);
    for (int R0 = tid / LPR + SROWS * M_STAGE; R0 < rtot; R0 += SROWS * M_STAGE) {
      stage_issue(R0);
      stage_store();
    }
  }
  if (bl_mine) bl[bl_l - 1][bl_u] = bl_ok ? bl_v : T(0);
  __syncthreads();  // weights, biases and the first tile's a_1 in LDS

  // the product of job jj over K inputs (a multiple of 4, at most the
  // 16-padded width, past which both sides are zero): lane (r, g) feeds
  // unit 16 ub + r and tile row 16 sb + r with input k + g.  TR reads the
  // staged weights transposed (the delta products W^T delta).
  int cur = 0;
  auto product = [&](auto tr, int jj, const T* w, int wp, int K) {
    constexpr bool TR = decltype(tr)::value;
    typename M::acc_t acc{};
    const T* h = &hs[cur][sblk(jj) + r][g];
    const T* wr = TR ? w + g * wp + unit(jj) : w + unit(jj) * wp + g;
    const int ws = TR ? wp : 1;  // weight stride per input
    // 32 inputs at a time: all their operands are read, then the products
    // run (the other waves of the SIMD cover the read latency); then 16,
    // then single steps of 4
    const int K32 = K & ~31, K16 = K & ~15;
    int k = 0;
    for (; k < K32; k += 32) {
      T xa[8], wb[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        wb[i] = wr[(k + 4 * i) * ws];
        xa[i] = h[k + 4 * i];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) acc = M::mma(xa[i], wb[i], acc);
      // keep the reads ahead of the products (the scheduler would otherwise
      // pair each read with its product and wait on it)
      __builtin_amdgcn_sched_group_barrier(0x100, 16, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    }
    if (k < K16) {
      T xa[4], wb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        wb[i] = wr[(k + 4 * i) * ws];
        xa[i] = h[k + 4 * i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) acc = M::mma(xa[i], wb[i], acc);
    }
    for (int k = K16; k < K; k += 4) acc = M::mma(h[k], wr[k * ws], acc);
    return acc;
  };
  using fwd_t = std::integral_constant<bool, false>;
  using bwd_t = std::integral_constant<bool, true>;

  for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int s0 = t * TS, rem = p.B - s0;
    if (t != (int)blockIdx.x) {
      layer1(t);
      __syncthreads();
    }

    // ---- layers 2..L: z_l = W_l a_{l-1} + b_l; at l = L the output delta.
    // Each job's activation follows its own product, so one wave's
    // activation arithmetic overlaps the other waves' matrix work.
#pragma unroll
    for (int l = 2; l <= L; ++l) {
      const int N = p.dims[l], K = (p.dims[l - 1] + 3) & ~3;
      const int wp = p.wp[l - 1];
      const T* w = wl + p.woff[l - 1];
      const __amdgpu_buffer_rsrc_t ores = rsrc(l < L ? p.A[l - 1] : p.D[l - 1]);
      const int lda = (int)p.lda[l - 1];
      with_act(p.acts[l - 1], [&](auto act) {
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
          if (!has_job(jj, N)) break;
          const typename M::acc_t acc = product(fwd_t{}, jj, w, wp, K);
          const int u = unit(jj), rw = row(jj);
          const unsigned vb = SZ * (unsigned)(rw * lda + u);
          const T b = bl[l - 1][u];
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const bool ok = u < N && rw + RS * v < rem;
            const unsigned so = SZ * (unsigned)((s0 + RS * v) * lda);
            T a, f;
            act_eval(decltype(act)::value, acc[v] + b, a, f);
            if (l < L) {
              a = ok ? a : T(0);
              M::store(a, ores, ok ? vb : MEDIUM_OOB, so);
              hs[cur ^ 1][rw + RS * v][u] = a;
              fp[l - 1][jj][v] = f;
            } else {
              const T d = ok ? (a - py[jj][v]) * f : T(0);
              M::store(d, ores, ok ? vb : MEDIUM_OOB, so);
              hs[cur ^ 1][rw + RS * v][u] = d;
            }
          }
        }
      });
      if (l == L) load_y(t + gridDim.x);
      cur ^= 1;
      __syncthreads();
    }

    // ---- hidden deltas, l = L-1 .. 1: (W_{l+1}^T delta_{l+1}) * f'(z_l).
    // Phases so far flipped the LDS buffers 2L - 3 times, so layer 1's delta
    // reads buffer 1 and the next tile's layer 1 may write buffer 0 without
    // another barrier.
#pragma unroll
    for (int l = L - 1; l >= 1; --l) {
      const int N = p.dims[l], K = (p.dims[l + 1] + 3) & ~3;
      const int wp = p.wp[l];
      const T* w = wl + p.woff[l];
      const __amdgpu_buffer_rsrc_t dres = rsrc(p.D[l - 1]);
      const int lda = (int)p.lda[l - 1];
#pragma unroll
      for (int jj = 0; jj < NJ; ++jj) {
        if (!has_job(jj, N)) break;
        const typename M::acc_t acc = product(bwd_t{}, jj, w, wp, K);
        const int u = unit(jj), rw = row(jj);
        const unsigned vb = SZ * (unsigned)(rw * lda + u);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const bool ok = u < N && rw + RS * v < rem;
          const T d = ok ? acc[v] * fp[l - 1][jj][v] : T(0);
          M::store(d, dres, ok ? vb : MEDIUM_OOB, SZ * (unsigned)((s0 + RS * v) * lda));
          if (l > 1) hs[cur ^ 1][rw + RS * v][u] = d;
        }
      }
      cur ^= 1;
      if (l > 1) __syncthreads();
    }
  }
}

// 16-sample blocks per tile: enough for one tile per CU where that takes at
// most 3 (3 blocks of 128 padded units fill LDS beside the largest weights);
// bigger batches run several rounds of tiles.  fp64 tiles are one block (the
// fp64 weights leave room for no more).
static int medium_tile_blocks(int B, int ncu, int esz) {
  if (esz == 8) return 1;
  const int blocks = (B + 15) / 16;
  const int nsb = (blocks + ncu - 1) / ncu;
  return nsb < 1 ? 1 : nsb > 3 ? 3 : nsb;
}

template <class T, int NSB>
static hipError_t launch_nsb(const MediumParamsT<T>& p, dim3 grid, hipStream_t s) {
  switch (p.L) {
    case 2: return launch_k(medium_kernel<T, NSB, 2>, grid, M_THREADS, 0, s, p);
    case 3: return launch_k(medium_kernel<T, NSB, 3>, grid, M_THREADS, 0, s, p);
    default: return launch_k(medium_kernel<T, NSB, 4>, grid, M_THREADS, 0, s, p);
  }
}

template <class T>
hipError_t launch_medium(const MediumParamsT<T>& p, int ncu, hipStream_t s) {
  if (p.L < 2 || p.L > MEDIUM_MAX_LAYERS) return hipErrorInvalidValue;
  const int nsb = medium_tile_blocks(p.B, ncu, (int)sizeof(T));
  const int ntiles = (p.B + 16 * nsb - 1) / (16 * nsb);
  const dim3 grid(ntiles < ncu ? ntiles : ncu);
  if constexpr (sizeof(T) == 8) {
    return launch_nsb<T, 1>(p, grid, s);
  } else {
    switch (nsb) {
      case 1: return launch_nsb<T, 1>(p, grid, s);
      case 2: return launch_nsb<T, 2>(p, grid, s);
      default: return launch_nsb<T, 3>(p, grid, s);
    }
  }
}

template hipError_t launch_medium<float>(const MediumParamsT<float>&, int, hipStream_t);
template hipError_t launch_medium<double>(const MediumParamsT<double>&, int, hipStream_t);

}  // namespace nf
