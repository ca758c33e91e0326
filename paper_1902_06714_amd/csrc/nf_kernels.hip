// Kernels for mini-batch MLP training on gfx950 (CDNA4), in fp32 (the
// paper's default real kind) and fp64 (its real64 kind).
//
// Every layer step of the method is one tiled contraction on the matrix cores
// (v_mfma_f32_32x32x2_f32, or v_mfma_f64_16x16x4_f64) with the rest of the
// step fused into its epilogue:
//   forward     Z = A_{l-1} W_l^T, + b_l, activation and its derivative
//               (section 3.2, Eq. 2; f' is kept for back-propagation)
//   output      delta_L = (f(z_L) - y) f'(z_L)   (section 3.3)
//   backward    delta_l = (delta_{l+1} W_{l+1}) * f'(z_l)   (section 3.3)
//   tendencies  G_l = delta_l^T A_{l-1} and g_l = column sums of delta_l,
//               summed over the batch in a fixed order, with the SGD step
//               W_l' = W_l - (eta/B) G_l fused in when the batch is one piece
//               (sections 3.3-3.5); the updated parameters go to a second
//               buffer, so every kernel leaves its inputs untouched
// Reductions run in a fixed order (each accumulator walks k upwards; pieces
// of a split batch are added in piece order), so results are bitwise
// reproducible from run to run.  No floating-point atomics are used.
#include "nf_act.h"
#include "nf_internal.h"
#include "nf_split.h"

namespace nf {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef double doublex4 __attribute__((ext_vector_type(4)));

// The matrix-core instruction of each element type, as the contraction uses
// it: a BLK x BLK block of C per instruction, KS values of k per instruction.
// Lane l supplies A(a_row(l), k0 + k_of(l)) and B(k0 + k_of(l), a_row(l)), and
// accumulator register v of lane l holds C(row(v, l), col(l)) of the block.
template <class T>
struct Mma;

template <>
struct Mma<float> {
  static constexpr int BLK = 32, KS = 2, NACC = 16;
  typedef floatx16 acc_t;
  __device__ static __forceinline__ acc_t mma(float a, float b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ int a_row(int l) { return l & 31; }
  __device__ static __forceinline__ int k_of(int l) { return l >> 5; }
  __device__ static __forceinline__ int row(int v, int l) {
    return 8 * (v >> 2) + 4 * (l >> 5) + (v & 3);
  }
  __device__ static __forceinline__ int col(int l) { return l & 31; }
};

template <>
struct Mma<double> {
  static constexpr int BLK = 16, KS = 4, NACC = 4;
  typedef doublex4 acc_t;
  __device__ static __forceinline__ acc_t mma(double a, double b, acc_t c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ int a_row(int l) { return l & 15; }
  __device__ static __forceinline__ int k_of(int l) { return l >> 4; }
  __device__ static __forceinline__ int row(int v, int l) { return 4 * v + (l >> 4); }
  __device__ static __forceinline__ int col(int l) { return l & 15; }
};

__device__ __forceinline__ float fma_t(float a, float b, float c) { return fmaf(a, b, c); }
__device__ __forceinline__ double fma_t(double a, double b, double c) { return fma(a, b, c); }

// 16 bytes of elements, the unit of a vector load
template <class T>
struct alignas(16) Vec16 {
  static constexpr int N = 16 / sizeof(T);
  T e[N];
};

// Global -> register -> LDS staging of one R x BK operand tile X(r, k),
// r in [r0, r0 + R), k in [k0, k0 + BK).  In LDS the tile is k-major,
// lds[k * SR + r], which is the order the MFMA operand reads want.  The row
// pitch SR is R + 4 when the tile arrives mn-contiguous (16-byte stores stay
// aligned) and R + 2 when it arrives k-contiguous: each thread then scatters
// a 16-byte load over 4 consecutive k rows, and with R + 2 the four row groups
// a wave writes at once fall in different banks (R + 4 put rows k and k + 8
// in the same ones).
// KC: k is the contiguous index in memory (X[r*ld + k]), else X[k*ld + r].
// VEC: rows are 16-byte aligned with a pitch that is a multiple of VW and the
// pitch padding is zero, so aligned 16-byte loads are safe.
// The loads go through a buffer resource based at the tile's first row (KC)
// or the stage's first k (otherwise), so offsets stay small for any matrix;
// elements outside the matrix or past the piece's k range are read at an
// offset past the buffer, which returns zeros without a memory access.  So
// every load is unconditional, stages past the end included.
constexpr unsigned TILE_OOB = 0x7ffffff0u;   // the buffers' length in bytes

template <class T, int R, int BK, int NT, bool KC, bool VEC>
struct TileLoader {
  static constexpr int VW = Vec16<T>::N;
  static constexpr int SR = R + (KC ? 2 : 4);
  static constexpr int NV = VEC ? (R * BK / VW) / NT : (R * BK) / NT;
  static_assert(VEC ? (R * BK / VW) % NT == 0 : (R * BK) % NT == 0, "tile not divisible");
  Vec16<T> v[VEC ? NV : 1];
  T s[VEC ? 1 : NV];

  __device__ __forceinline__ void load(const T* __restrict__ X, int64_t ld, int rmax, int kend,
                                       int r0, int k0, int tid) {
    const T* base = KC ? X + (int64_t)r0 * ld : X + (int64_t)k0 * ld;
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, (int)TILE_OOB, 0x00020000);
    const int ldi = (int)ld;
    if constexpr (VEC) {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int q = tid + i * NT;
        int r, k;
        if constexpr (KC) {
          r = q / (BK / VW);
          k = (q % (BK / VW)) * VW;
        } else {
          k = q / (R / VW);
          r = (q % (R / VW)) * VW;
        }
        const int gr = r0 + r, gk = k0 + k;
        const int e = KC ? r * ldi + gk : k * ldi + gr;
        const unsigned off = (gr < rmax && gk < kend) ? (unsigned)e * (unsigned)sizeof(T) : TILE_OOB;
        v[i] = __builtin_bit_cast(Vec16<T>, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
      }
    } else {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int q = tid + i * NT;
        int r, k;
        if constexpr (KC) {
          r = q / BK;
          k = q % BK;
        } else {
          k = q / R;
          r = q % R;
        }
        const int gr = r0 + r, gk = k0 + k;
        const int e = KC ? r * ldi + gk : k * ldi + gr;
        const unsigned off = (gr < rmax && gk < kend) ? (unsigned)e * (unsigned)sizeof(T) : TILE_OOB;
        if constexpr (sizeof(T) == 4)
          s[i] = __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0));
        else
          s[i] = __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0));
      }
    }
  }

  __device__ __forceinline__ void store(T* lds, int tid) const {
    if constexpr (VEC) {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int q = tid + i * NT;
        if constexpr (KC) {
          const int r = q / (BK / VW), k = (q % (BK / VW)) * VW;
#pragma unroll
          for (int c = 0; c < VW; ++c) lds[(k + c) * SR + r] = v[i].e[c];
        } else {
          const int k = q / (R / VW), r = (q % (R / VW)) * VW;
          *reinterpret_cast<Vec16<T>*>(lds + k * SR + r) = v[i];
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int e = tid + i * NT;
        int r, k;
        if constexpr (KC) {
          r = e / BK;
          k = e % BK;
        } else {
          k = e / R;
          r = e % R;
        }
        lds[k * SR + r] = s[i];
      }
    }
  }
};

// C[BM x BN] tile per workgroup; (BM/WM) x (BN/WN) waves, each owning a
// WM x WN sub-tile made of BLK x BLK matrix-core blocks.  grid = (M tiles,
// N tiles, pieces of the k range).
template <class T, int BM, int BN, int BK, int WM, int WN, int PD, bool AKC, bool BKC, bool AV,
          bool BV, int EPI>
__device__ __forceinline__ void gemm_tile(const GemmParamsT<T>& p, int bx, int by, int bz) {
  using MM = Mma<T>;
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  constexpr int TM = WM / MM::BLK, TN = WN / MM::BLK;
  // LDS row pitches, as in TileLoader
  constexpr int SA = BM + (AKC ? 2 : 4), SB = BN + (BKC ? 2 : 4);
  __shared__ __attribute__((aligned(16))) T As[2][BK * SA];
  __shared__ __attribute__((aligned(16))) T Bs[2][BK * SB];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = (wave % (BM / WM)) * WM;
  const int wn = (wave / (BM / WM)) * WN;
  const int m0 = bx * BM;
  const int n0 = by * BN;

  // k range of this piece
  int kbeg = 0, kend = p.K;
  if constexpr (EPI == EPI_DW_SGD || EPI == EPI_DW_PARTIAL || EPI == EPI_FWD_PIECE) {
    const int z = bz;
    const int shard = z / p.nsub, sub = z % p.nsub;
    const int sb = shard * p.shard_len;
    kbeg = sb + sub * p.sub_len;
    kend = min(kbeg + p.sub_len, sb + p.shard_len);
  }
  const bool do_bias = (EPI == EPI_DW_SGD || EPI == EPI_DW_PARTIAL) && by == 0;

  typename MM::acc_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < MM::NACC; ++v) acc[i][j][v] = T(0);
  T bsum = T(0);

  const int ntiles = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;

  // PD register stages of the operand tiles are in flight: stage t + 1 goes
  // to LDS while stage t is multiplied, and its registers then take stage
  // t + 1 + PD.  Stage s is held by register set s % PD; after the prologue
  // LDS holds stage 0, set k stage k (k >= 1) and set 0 stage PD.
  TileLoader<T, BM, BK, NT, AKC, AV> la[PD];
  TileLoader<T, BN, BK, NT, BKC, BV> lb[PD];
#pragma unroll
  for (int d = 0; d < PD; ++d) {
    la[d].load(p.A, p.lda, p.M, kend, m0, kbeg + d * BK, tid);
    lb[d].load(p.B, p.ldb, p.N, kend, n0, kbeg + d * BK, tid);
  }
  la[0].store(As[0], tid);
  lb[0].store(Bs[0], tid);
  la[0].load(p.A, p.lda, p.M, kend, m0, kbeg + PD * BK, tid);
  lb[0].load(p.B, p.ldb, p.N, kend, n0, kbeg + PD * BK, tid);
  __syncthreads();

  // the products of stage t, held in LDS buffer t & 1
  auto multiply = [&](int t) {
    const T* a_s = As[t & 1];
    const T* b_s = Bs[t & 1];
#pragma unroll
    for (int kk = 0; kk < BK; kk += MM::KS) {
      T av[TM], bv[TN];
      const int krow = kk + MM::k_of(lane);
#pragma unroll
      for (int i = 0; i < TM; ++i) av[i] = a_s[krow * SA + wm + i * MM::BLK + MM::a_row(lane)];
#pragma unroll
      for (int j = 0; j < TN; ++j) bv[j] = b_s[krow * SB + wn + j * MM::BLK + MM::a_row(lane)];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = MM::mma(av[i], bv[j], acc[i][j]);
    }
    if (do_bias && tid < BM) {
      // column sums of delta (the bias tendency), k in increasing order
#pragma unroll
      for (int kk = 0; kk < BK; ++kk) bsum += a_s[kk * SA + tid];
    }
  };

  // Whole groups of PD stages, every load unconditional (past the last stage
  // they read zeros): the compiler then waits for exactly the stage it needs.
  // The last stages follow the loop; their inputs are already requested.
  int t = 0;
  for (; t + PD <= ntiles; t += PD) {
#pragma unroll
    for (int d = 0; d < PD; ++d) {
      const int j = (d + 1) % PD;
      multiply(t + d);
      la[j].store(As[(t + d + 1) & 1], tid);
      lb[j].store(Bs[(t + d + 1) & 1], tid);
      la[j].load(p.A, p.lda, p.M, kend, m0, kbeg + (t + d + 1 + PD) * BK, tid);
      lb[j].load(p.B, p.ldb, p.N, kend, n0, kbeg + (t + d + 1 + PD) * BK, tid);
      __syncthreads();
    }
  }
#pragma unroll
  for (int d = 0; d < PD - 1; ++d) {
    if (t + d < ntiles) {
      const int j = (d + 1) % PD;
      multiply(t + d);
      if (t + d + 1 < ntiles) {
        la[j].store(As[(t + d + 1) & 1], tid);
        lb[j].store(Bs[(t + d + 1) & 1], tid);
      }
      __syncthreads();
    }
  }

  // Epilogue: accumulator register v of this lane holds row MM::row(v, lane)
  // and column MM::col(lane) of its block.
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + wn + j * MM::BLK + MM::col(lane);
      if (n >= p.N) continue;
      T bn = T(0);
      if constexpr (EPI == EPI_FWD_STASH || EPI == EPI_FWD_DELTA || EPI == EPI_FWD_OUT)
        bn = p.bias[n];
#pragma unroll
      for (int v = 0; v < MM::NACC; ++v) {
        const int m = m0 + wm + i * MM::BLK + MM::row(v, lane);
        if (m >= p.M) continue;
        const T c = acc[i][j][v];
        if constexpr (EPI == EPI_FWD_STASH) {
          T f, fp;
          act_eval(p.act, c + bn, f, fp);
          p.out0[(int64_t)m * p.ld0 + n] = f;
          p.out1[(int64_t)m * p.ld1 + n] = fp;
        } else if constexpr (EPI == EPI_FWD_DELTA) {
          T f, fp;
          act_eval(p.act, c + bn, f, fp);
          p.out0[(int64_t)m * p.ld0 + n] = (f - p.aux[(int64_t)m * p.ldaux + n]) * fp;
        } else if constexpr (EPI == EPI_FWD_OUT) {
          T f, fp;
          act_eval(p.act, c + bn, f, fp);
          p.out0[(int64_t)m * p.ld0 + n] = f;
        } else if constexpr (EPI == EPI_BWD) {
          p.out0[(int64_t)m * p.ld0 + n] = c * p.aux[(int64_t)m * p.ldaux + n];
        } else if constexpr (EPI == EPI_DW_SGD) {
          const int64_t o = (int64_t)m * p.ldw + n;
          p.out0[o] = c;
          p.W[o] = fma_t(-p.scale, c, p.Win[o]);
        } else {  // EPI_DW_PARTIAL, EPI_FWD_PIECE
          p.partial[(int64_t)bz * p.pstride + (int64_t)m * p.ld0 + n] = c;
        }
      }
    }
  }
  if (do_bias && tid < BM) {
    const int m = m0 + tid;
    if (m < p.M) {
      if constexpr (EPI == EPI_DW_SGD) {
        p.gbias[m] = bsum;
        p.bvec[m] = fma_t(-p.scale, bsum, p.bin[m]);
      } else if constexpr (EPI == EPI_DW_PARTIAL) {
        p.pbias[(int64_t)bz * p.M + m] = bsum;
      }
    }
  }
}


// One launch of one contraction: grid = (M tiles, N tiles, pieces of the k range).
template <class T, int BM, int BN, int BK, int WM, int WN, int PD, bool AKC, bool BKC, bool AV,
          bool BV, int EPI>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
gemm_kernel(const GemmParamsT<T> p) {
  gemm_tile<T, BM, BN, BK, WM, WN, PD, AKC, BKC, AV, BV, EPI>(p, blockIdx.x, blockIdx.y, blockIdx.z);
}

// One launch of several contractions of the same shape class (the tendency
// pieces of several layers): workgroup b belongs to the problem q with
// start[q] <= b < start[q + 1] and takes its tiles in the order of the
// single-problem grid (M tiles fastest, then N tiles, then pieces).
template <class T, int BM, int BN, int BK, int WM, int WN, int PD, bool AKC, bool BKC, bool AV,
          bool BV, int EPI>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
gemm_group_kernel(const GemmGroupT<T> g) {
  const int b = blockIdx.x;
  int q = 0;
#pragma unroll
  for (int i = 1; i < GEMM_GROUP_MAX; ++i) q += (i < g.n && b >= g.start[i]);
  const int r = b - g.start[q];
  const int mt = (g.p[q].M + BM - 1) / BM, nt = (g.p[q].N + BN - 1) / BN;
  const int z = r / (mt * nt), rem = r % (mt * nt);
  gemm_tile<T, BM, BN, BK, WM, WN, PD, AKC, BKC, AV, BV, EPI>(g.p[q], rem % mt, rem / mt, z);
}

// Sum of the per-piece tendencies in piece order, then the SGD step (from the
// parameters before the step into the other parameter buffer), for up to
// FOLD_GROUP_MAX layers per launch; workgroup b belongs to layer q with
// start[q] <= b < start[q + 1].
// The shard fold of one value: pieces q = s nsub + u (shard s, sub-piece u)
// in order, piece_s = ((p_{s,0} + p_{s,1}) + ...), total = ((piece_0 +
// piece_1) + ...).  The loads of a batch of NB pieces issue together before
// any is added (past the last piece a batch re-reads the last one and drops
// it), so a fold of up to NB pieces waits for memory once, not once per
// piece.  NB is the smallest of 4, 8, 16, 32 that holds every piece (32
// past that), so folds of few pieces (bandwidth-bound on large layers) read
// no extra bytes.
template <int NB, class T, class Get>
__device__ __forceinline__ T fold_pieces_nb(int nsub, int P, Get get) {
  T tot = T(0), piece = T(0);
  int u = 0;           // sub-piece within the current shard
  bool first = true;   // no shard added to the total yet
  auto batch = [&](int q0) {
    T v[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) v[i] = get(q0 + i < P ? q0 + i : P - 1);
    __builtin_amdgcn_sched_barrier(0);  // every load of the batch before the first add
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if (q0 + i < P) {
        piece = u == 0 ? v[i] : piece + v[i];
        if (++u == nsub) {
          tot = first ? piece : tot + piece;
          first = false;
          u = 0;
        }
      }
    }
  };
  // the first batch outside the loop (P >= 1): a loop head would wait for
  // the loads issued before it
  batch(0);
  for (int q0 = NB; q0 < P; q0 += NB) batch(q0);
  return tot;
}

template <class T, class Get>
__device__ __forceinline__ T fold_pieces(int nshards, int nsub, Get get) {
  const int P = nshards * nsub;
  if (P <= 4) return fold_pieces_nb<4, T>(nsub, P, get);
  if (P <= 8) return fold_pieces_nb<8, T>(nsub, P, get);
  if (P <= 16) return fold_pieces_nb<16, T>(nsub, P, get);
  return fold_pieces_nb<32, T>(nsub, P, get);
}

template <class T>
__global__ void fold_sgd_kernel(const FoldGroupT<T> g) {
  const int b = blockIdx.x;
  int q = 0;
#pragma unroll
  for (int i = 1; i < FOLD_GROUP_MAX; ++i) q += (i < g.n && b >= g.start[i]);
  const FoldLayerT<T>& f = g.l[q];
  const int64_t idx = (int64_t)(b - g.start[q]) * blockDim.x + threadIdx.x;
  const int64_t nw = (int64_t)f.M * f.N;
  const int nshards = g.nshards, nsub = f.nsub;
  if (idx < nw) {
    const int m = (int)(idx / f.N), n = (int)(idx % f.N);
    const int64_t o = (int64_t)m * f.ldw + n;
    const T w_old = f.Win[o];
    const T tot = fold_pieces<T>(nshards, nsub,
                                 [&](int q) { return f.partial[(int64_t)q * f.pstride + o]; });
    f.G[o] = tot;
    f.W[o] = fma_t(-g.scale, tot, w_old);
  } else if (idx < nw + f.M) {
    const int m = (int)(idx - nw);
    const T b_old = f.bin[m];
    const T tot = fold_pieces<T>(nshards, nsub,
                                 [&](int q) { return f.pbias[(int64_t)q * f.M + m]; });
    f.gbias[m] = tot;
    f.b[m] = fma_t(-g.scale, tot, b_old);
  }
}

// Operand stages in flight per tile shape (measured).  The 128 x 128 tile
// runs one workgroup per CU on large problems and needs the depth; the
// 64 x 64 tile serves small grids, where extra stages cost registers and so
// workgroups per CU, which hide the memory latency better.
constexpr int PD_128 = 4;
constexpr int PD_64 = 2;

template <class T, int BM, int BN, int BK, int WM, int WN, int PD, bool AKC, bool BKC, bool AV,
          bool BV, int EPI>
static hipError_t launch_one(int nsplit, const GemmParamsT<T>& p, hipStream_t s) {
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  dim3 grid((p.M + BM - 1) / BM, (p.N + BN - 1) / BN, nsplit);
  return launch_k(gemm_kernel<T, BM, BN, BK, WM, WN, PD, AKC, BKC, AV, BV, EPI>, grid, NT, 0, s,
                  p);
}

template <class T, int BM, int BN, int BK, int WM, int WN, int PD>
static hipError_t dispatch_tile(int epi, bool akc, bool bkc, bool av, bool bv, int nsplit,
                                const GemmParamsT<T>& p, hipStream_t s) {
#define NF_CASE(AKC, BKC, AV, BV, E)                                     \
  if (akc == AKC && bkc == BKC && av == AV && bv == BV && epi == E)      \
    return launch_one<T, BM, BN, BK, WM, WN, PD, AKC, BKC, AV, BV, E>(nsplit, p, s);
  // forward: A = activations [m][k], B(k, n) = W[n][k]
  NF_CASE(true, true, true, true, EPI_FWD_STASH)
  NF_CASE(true, true, false, true, EPI_FWD_STASH)
  NF_CASE(true, true, true, true, EPI_FWD_DELTA)
  NF_CASE(true, true, false, true, EPI_FWD_DELTA)
  NF_CASE(true, true, true, true, EPI_FWD_OUT)
  NF_CASE(true, true, false, true, EPI_FWD_OUT)
  NF_CASE(true, true, true, true, EPI_FWD_PIECE)
  NF_CASE(true, true, false, true, EPI_FWD_PIECE)
  // backward: A = delta [m][k], B(k, n) = W[k][n]
  NF_CASE(true, false, true, true, EPI_BWD)
  // tendencies: A(m, k) = delta[k][m], B(k, n) = activations[k][n] (the
  // tendency pieces go through launch_dw_partial_group)
  NF_CASE(false, false, true, true, EPI_DW_SGD)
  NF_CASE(false, false, true, false, EPI_DW_SGD)
#undef NF_CASE
  return hipErrorInvalidValue;
}

template <class T>
hipError_t launch_gemm(int epi, int tile, bool a_kcontig, bool b_kcontig, bool a_vec, bool b_vec,
                       int nsplit, const GemmParamsT<T>& p, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0 || nsplit <= 0) return hipErrorInvalidValue;
  // The epilogues that work on pieces of the k range read an operand that is
  // k-contiguous and loaded 16 bytes at a time only if every piece starts on
  // a whole BK stage (nf_split.h): a piece start off that grid would make
  // the last vector of the piece before it read into this piece and past the
  // operand's rows.  (The tendency pieces split the batch, which is not the
  // contiguous index of either of their operands, so any cut is safe there.)
  if (epi == EPI_FWD_PIECE || epi == EPI_DW_SGD || epi == EPI_DW_PARTIAL) {
    if (p.nsub <= 0 || nsplit % p.nsub != 0) return hipErrorInvalidValue;
    if (((a_kcontig && a_vec) || (b_kcontig && b_vec)) &&
        !k_pieces_aligned(nsplit / p.nsub, p.shard_len, p.nsub, p.sub_len))
      return hipErrorInvalidValue;
  }
  // The 128 x 128 tile runs 8 waves of 64 x 32 (two per SIMD, so one
  // wave's LDS reads and barrier waits overlap the other's matrix work).
  constexpr int WN128 = 32;
  // element offsets inside one buffer-based tile stay below TILE_OOB bytes
  if ((int64_t)128 * (p.lda > p.ldb ? p.lda : p.ldb) * (int64_t)sizeof(T) >= (int64_t)TILE_OOB)
    return hipErrorInvalidValue;
  if (tile == TILE_128x128)
    return dispatch_tile<T, 128, 128, 16, 64, WN128, PD_128>(epi, a_kcontig, b_kcontig, a_vec,
                                                            b_vec, nsplit, p, s);
  return dispatch_tile<T, 64, 64, 16, 32, 32, PD_64>(epi, a_kcontig, b_kcontig, a_vec, b_vec,
                                                    nsplit, p, s);
}

template hipError_t launch_gemm<float>(int, int, bool, bool, bool, bool, int,
                                       const GemmParamsT<float>&, hipStream_t);
template hipError_t launch_gemm<double>(int, int, bool, bool, bool, bool, int,
                                        const GemmParamsT<double>&, hipStream_t);

const char* gemm_name(int epi, int tile, int dtype) {
  static const char* names[2][2][7] = {
      {{"gemm_fwd_stash_128x128", "gemm_fwd_delta_128x128", "gemm_fwd_out_128x128",
        "gemm_bwd_128x128", "gemm_dw_sgd_128x128", "gemm_dw_partial_128x128",
        "gemm_fwd_piece_128x128"},
       {"gemm_fwd_stash_64x64", "gemm_fwd_delta_64x64", "gemm_fwd_out_64x64", "gemm_bwd_64x64",
        "gemm_dw_sgd_64x64", "gemm_dw_partial_64x64", "gemm_fwd_piece_64x64"}},
      {{"gemm64_fwd_stash_128x128", "gemm64_fwd_delta_128x128", "gemm64_fwd_out_128x128",
        "gemm64_bwd_128x128", "gemm64_dw_sgd_128x128", "gemm64_dw_partial_128x128",
        "gemm64_fwd_piece_128x128"},
       {"gemm64_fwd_stash_64x64", "gemm64_fwd_delta_64x64", "gemm64_fwd_out_64x64",
        "gemm64_bwd_64x64", "gemm64_dw_sgd_64x64", "gemm64_dw_partial_64x64",
        "gemm64_fwd_piece_64x64"}}};
  if (epi < 0 || epi > 6 || tile < 0 || tile > 1 || dtype < 0 || dtype > 1) return "gemm";
  return names[dtype][tile][epi];
}

// The forward epilogue on the sum of a split contraction's pieces (piece
// order), one thread per (m, n), n fastest.
template <class T, int EPI>
__global__ void fwd_fold_kernel(const FwdFoldParamsT<T> f) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)f.M * f.N) return;
  const int m = (int)(idx / f.N), n = (int)(idx % f.N);
  const int64_t o = (int64_t)m * f.ldp + n;
  // the bias and the target requested with the pieces, all before the first use
  const T bias = f.bias[n];
  const T y = EPI == EPI_FWD_DELTA ? f.aux[(int64_t)m * f.ldaux + n] : T(0);
  const T z = fold_pieces<T>(f.nsplit, 1,
                             [&](int q) { return f.partial[(int64_t)q * f.pstride + o]; });
  T a, fp;
  act_eval(f.act, z + bias, a, fp);
  if constexpr (EPI == EPI_FWD_STASH) {
    f.out0[(int64_t)m * f.ld0 + n] = a;
    f.out1[(int64_t)m * f.ld1 + n] = fp;
  } else if constexpr (EPI == EPI_FWD_DELTA) {
    f.out0[(int64_t)m * f.ld0 + n] = (a - y) * fp;
  } else {
    f.out0[(int64_t)m * f.ld0 + n] = a;
  }
}

template <class T>
hipError_t launch_fwd_fold(int epi, const FwdFoldParamsT<T>& f, hipStream_t s) {
  const int64_t total = (int64_t)f.M * f.N;
  if (total <= 0 || f.nsplit < 1) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((total + 255) / 256));
  if (epi == EPI_FWD_STASH)
    return launch_k(fwd_fold_kernel<T, EPI_FWD_STASH>, grid, 256, 0, s, f);
  else if (epi == EPI_FWD_DELTA)
    return launch_k(fwd_fold_kernel<T, EPI_FWD_DELTA>, grid, 256, 0, s, f);
  else if (epi == EPI_FWD_OUT)
    return launch_k(fwd_fold_kernel<T, EPI_FWD_OUT>, grid, 256, 0, s, f);
  return hipErrorInvalidValue;
}

template hipError_t launch_fwd_fold<float>(int, const FwdFoldParamsT<float>&, hipStream_t);
template hipError_t launch_fwd_fold<double>(int, const FwdFoldParamsT<double>&, hipStream_t);

template <class T>
hipError_t launch_fold_sgd(FoldGroupT<T> g, hipStream_t s) {
  if (g.n < 1 || g.n > FOLD_GROUP_MAX) return hipErrorInvalidValue;
  const int threads = FOLD_THREADS;
  g.start[0] = 0;
  for (int q = 0; q < g.n; ++q) {
    const int64_t elems = (int64_t)g.l[q].M * g.l[q].N + g.l[q].M;
    g.start[q + 1] = g.start[q] + (int)((elems + threads - 1) / threads);
  }
  for (int q = g.n + 1; q <= FOLD_GROUP_MAX; ++q) g.start[q] = g.start[g.n];
  return launch_k(fold_sgd_kernel<T>, dim3((unsigned)g.start[g.n]), threads, 0, s, g);
}

template hipError_t launch_fold_sgd<float>(FoldGroupT<float>, hipStream_t);
template hipError_t launch_fold_sgd<double>(FoldGroupT<double>, hipStream_t);

template <class T, int BM, int BN, int WM, int WN, int PD, bool BV>
static hipError_t launch_group(GemmGroupT<T> g, const int* nsplit, hipStream_t s) {
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  g.start[0] = 0;
  for (int q = 0; q < g.n; ++q) {
    const int mt = (g.p[q].M + BM - 1) / BM, nt = (g.p[q].N + BN - 1) / BN;
    g.start[q + 1] = g.start[q] + mt * nt * nsplit[q];
  }
  for (int q = g.n + 1; q <= GEMM_GROUP_MAX; ++q) g.start[q] = g.start[g.n];
  return launch_k(
      gemm_group_kernel<T, BM, BN, 16, WM, WN, PD, false, false, true, BV, EPI_DW_PARTIAL>,
      dim3((unsigned)g.start[g.n]), NT, 0, s, g);
}

template <class T>
hipError_t launch_dw_partial_group(int tile, bool b_vec, const GemmGroupT<T>& g,
                                   const int* nsplit, hipStream_t s) {
  if (g.n < 1 || g.n > GEMM_GROUP_MAX) return hipErrorInvalidValue;
  // the group kernels read both operands mn-contiguous (the batch, which the
  // pieces split, is their row index), so no piece alignment is needed
  for (int q = 0; q < g.n; ++q) {
    if (g.p[q].M <= 0 || g.p[q].N <= 0 || nsplit[q] <= 0) return hipErrorInvalidValue;
    if (g.p[q].nsub <= 0 || nsplit[q] % g.p[q].nsub != 0) return hipErrorInvalidValue;
    const int64_t ld = g.p[q].lda > g.p[q].ldb ? g.p[q].lda : g.p[q].ldb;
    if ((int64_t)128 * ld * (int64_t)sizeof(T) >= (int64_t)TILE_OOB) return hipErrorInvalidValue;
  }
  // the tiles and stage depths of launch_gemm
  if (tile == TILE_128x128)
    return b_vec ? launch_group<T, 128, 128, 64, 32, PD_128, true>(g, nsplit, s)
                 : launch_group<T, 128, 128, 64, 32, PD_128, false>(g, nsplit, s);
  return b_vec ? launch_group<T, 64, 64, 32, 32, PD_64, true>(g, nsplit, s)
               : launch_group<T, 64, 64, 32, 32, PD_64, false>(g, nsplit, s);
}

template hipError_t launch_dw_partial_group<float>(int, bool, const GemmGroupT<float>&, const int*,
                                                   hipStream_t);
template hipError_t launch_dw_partial_group<double>(int, bool, const GemmGroupT<double>&,
                                                    const int*, hipStream_t);

}  // namespace nf
