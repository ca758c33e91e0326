// Kernels for contractions one side of which is a layer of at most
// SKINNY_MAX_UNITS units, e.g. the 100-unit layers of a 784-100-100-10
// network: the tendency pieces in fp32 and fp64, and the layer-1 forward
// pieces in fp32.
//
// Tendency pieces (section 3.3: dC/dW_l = delta_l^T a_{l-1}, dC/db_l = the
// column sums of delta_l, each over one piece of the batch), fp32:
//
// Both operands are sample-major (delta_l[s][u], a_{l-1}[s][n]) and the sum
// runs over samples, so a 16-byte load gives a lane 4 consecutive units (or
// inputs) of one sample.  The kernel takes them straight from global memory
// into matrix-core operands, with no LDS staging and no barrier in the loop:
// in a 16x16x4 product lane (r, g) supplies row r of A and column r of B at
// input index g, so the 4 values of a lane's vector go to 4 different
// products.  Unit 4 r + e of a segment of 64 units is row r of unit block e;
// a layer's last units take a segment of 32 (8-byte loads, 2 blocks) and / or
// of 16 (4-byte loads, 1 block), so a layer of d units costs ceil(d / 16)
// blocks (7 for 100 units).  The inputs are cut the same way: tiles of 64
// (4 blocks), the last tile ceil(rest / 16) blocks.  Input index g of the
// products is sample 4 j + g of k-step j.  A wave holds every (unit block,
// input block) of its tile and per k-step of 4 samples issues one load per
// segment of each side (a 4 rows x 256 bytes pattern for a 64-wide
// segment).  SKINNY_PD k-steps of loads are in flight.
//
// A workgroup of 4 waves owns one (piece, input tile): wave w takes the w-th
// quarter of the piece's k-steps, and the four partial sums are added
// through LDS in wave order at the end, four unit blocks at a time.  A
// tile-0 workgroup also sums the delta columns (the bias tendency): each
// lane over its samples, then over the 4 lanes of a unit, then over the
// waves.
//
// Workgroups go round robin over the 8 XCDs (workgroup b runs on XCD b mod
// 8).  XCD x takes pieces x, x + 8, ... of a layer, each with all of its
// input tiles one after another, so a piece's delta rows are fetched into
// that XCD's L2 once.
//
// The per-piece sums land in the same [piece][M][ld0] + [piece][M] layout as
// the general tendency pieces, and fold_sgd_kernel folds them in piece order.
#include <atomic>

#include "nf_internal.h"

namespace nf {

typedef float floatx4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int SK_NT = 256;                 // 4 waves
constexpr int SK_TN = SKINNY_TILE_F32;     // inputs per tile
constexpr unsigned SK_OOB = 0x7ffffff0u;   // buffer length: offsets past it read 0
static_assert(SKINNY_MAX_UNITS <= 128, "at most 8 unit blocks");

__device__ __forceinline__ __amdgpu_buffer_rsrc_t sk_rsrc(const float* base) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, (int)SK_OOB, 0x00020000);
}

__device__ __forceinline__ floatx4 sk_load(__amdgpu_buffer_rsrc_t rs, unsigned off) {
  return __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
}

typedef float floatx2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ floatx2 sk_load2(__amdgpu_buffer_rsrc_t rs, unsigned off) {
  return __builtin_bit_cast(floatx2, __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0));
}
__device__ __forceinline__ float sk_load1(__amdgpu_buffer_rsrc_t rs, unsigned off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0));
}

// The blocks of one side (units or inputs) of a workgroup's tile: S4
// segments of 64 rows read with 16-byte loads (row 4 r + e of a segment is
// row r of its block e), then S2 <= 1 segment of 32 rows read with 8-byte
// loads (row 2 r + e: block e), then S1 <= 1 segment of 16 rows read with
// 4-byte loads (row r).  A side of d rows takes ceil(d / 16) blocks.
template <int S4, int S2, int S1>
struct SkSide {
  static constexpr int NB = 4 * S4 + 2 * S2 + S1;
  static constexpr int B2 = 64 * S4, B1 = 64 * S4 + 32 * S2;   // first rows of the segments
  // row of block b that lane row r supplies
  __device__ static int row(int b, int r) {
    if (b < 4 * S4) return 64 * (b >> 2) + 4 * r + (b & 3);
    if (b < 4 * S4 + 2 * S2) return B2 + 2 * r + (b - 4 * S4);
    return B1 + r;
  }
  struct Regs {
    floatx4 v4[S4 > 0 ? S4 : 1];
    floatx2 v2;
    float v1;
  };
  // one sample row's values of this lane: rows < lim are read at byte
  // offset base + 4 row; ok false reads zeros
  __device__ static void load(Regs& g, __amdgpu_buffer_rsrc_t rs, unsigned base, int r, int lim,
                              bool ok) {
#pragma unroll
    for (int i = 0; i < S4; ++i) {
      const int e = 64 * i + 4 * r;
      g.v4[i] = sk_load(rs, ok && e < lim ? base + 4u * (unsigned)e : SK_OOB);
    }
    if constexpr (S2 > 0) {
      const int e = B2 + 2 * r;
      g.v2 = sk_load2(rs, ok && e < lim ? base + 4u * (unsigned)e : SK_OOB);
    }
    if constexpr (S1 > 0) {
      const int e = B1 + r;
      g.v1 = sk_load1(rs, ok && e < lim ? base + 4u * (unsigned)e : SK_OOB);
    }
  }
  // the value of block b
  __device__ static float at(const Regs& g, int b) {
    if (b < 4 * S4) return g.v4[b >> 2][b & 3];
    if (b < 4 * S4 + 2 * S2) return g.v2[b - 4 * S4];
    return g.v1;
  }
};

// One workgroup's (piece, input tile): unit side U against input side X.
template <class U, class X>
__device__ __forceinline__ void skinny_tile(const GemmParamsT<float>& p, int piece, int tile,
                                            floatx4 (*red)[16][64], float (*bred)[SKINNY_MAX_UNITS]) {
  constexpr int NU = U::NB, NX = X::NB;
  const int M = p.M, N = p.N;
  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index, known to the compiler as uniform: the k-steps and so
  // the buffer resources stay in scalar registers
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, gq = lane >> 4;
  const int n0 = tile * SK_TN;
  const bool do_bias = tile == 0;

  const int shard = piece / p.nsub, sub = piece % p.nsub;
  const int sb = shard * p.shard_len;
  const int kbeg = sb + sub * p.sub_len;
  const int kend = min(kbeg + p.sub_len, sb + p.shard_len);
  const int nks = kend > kbeg ? (kend - kbeg + 3) >> 2 : 0;   // k-steps of 4 samples
  const int qk = (nks + 3) >> 2;
  const int j0 = min(nks, w * qk), j1 = min(nks, j0 + qk);
  const int lda = (int)p.lda, ldb = (int)p.ldb;
  const unsigned dbase = 4u * (unsigned)(gq * lda), xbase = 4u * (unsigned)(gq * ldb + n0);

  floatx4 acc[NU][NX];
#pragma unroll
  for (int a = 0; a < NU; ++a)
#pragma unroll
    for (int b = 0; b < NX; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};
  float bsum[NU];
#pragma unroll
  for (int a = 0; a < NU; ++a) bsum[a] = 0.f;

  struct Step {
    typename U::Regs d;
    typename X::Regs x;
  };
  // k-step j: samples kbeg + 4 j + gq; past j1 or kend the loads read zeros
  auto load = [&](Step& st, int j) {
    const int s0 = kbeg + 4 * j;
    const bool ok = j < j1 && s0 + gq < kend;
    U::load(st.d, sk_rsrc(p.A + (int64_t)s0 * lda), dbase, r, M, ok);
    X::load(st.x, sk_rsrc(p.B + (int64_t)s0 * ldb), xbase, r, N - n0, ok);
  };
  auto step = [&](const Step& st) {
#pragma unroll
    for (int a = 0; a < NU; ++a)
#pragma unroll
      for (int b = 0; b < NX; ++b)
        acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(U::at(st.d, a), X::at(st.x, b), acc[a][b],
                                                         0, 0, 0);
    if (do_bias) {
#pragma unroll
      for (int a = 0; a < NU; ++a) bsum[a] += U::at(st.d, a);
    }
  };

  // SKINNY_PD k-steps of loads in flight (one fewer with all 32 blocks,
  // whose accumulators fill half the registers); whole groups load
  // unconditionally (past the wave's range the loads read zeros), so each
  // wait is for exactly the k-step needed
  constexpr int PD = NU * NX > 28 ? SKINNY_PD - 1 : SKINNY_PD;
  Step st[PD];
#pragma unroll
  for (int d = 0; d < PD; ++d) load(st[d], j0 + d);
  int j = j0;
  for (; j + PD <= j1; j += PD) {
#pragma unroll
    for (int d = 0; d < PD; ++d) {
      step(st[d]);
      load(st[d], j + d + PD);
    }
  }
#pragma unroll
  for (int d = 0; d < PD - 1; ++d)
    if (j + d < j1) step(st[d]);

  if (do_bias) {
    // lanes r, r + 16, r + 32, r + 48 hold the same units
#pragma unroll
    for (int a = 0; a < NU; ++a) {
      float t = bsum[a];
      t += __shfl_xor(t, 16);
      t += __shfl_xor(t, 32);
      if (gq == 0) bred[w][U::row(a, r)] = t;
    }
  }

  // Unit blocks 4 c .. 4 c + 3 at a time: the input blocks b of a lane's
  // (unit block a, accumulator row v) go to LDS as one vector, slot
  // 4 (a - 4 c) + v; wave w then sums the slots of unit block 4 c + w over
  // the waves in wave order.  Accumulator row v of lane (r, gq) is row
  // 4 gq + v of the block (the unit), column r (the input).
  float* out = p.partial + (int64_t)piece * p.pstride;
#pragma unroll
  for (int c = 0; c < (NU + 3) / 4; ++c) {
    if (c > 0) __syncthreads();   // the previous blocks' sums are read
#pragma unroll
    for (int a = 4 * c; a < 4 * c + 4 && a < NU; ++a)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        floatx4 t = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int b = 0; b < NX; ++b) t[b] = acc[a][b][v];
        red[w][4 * (a - 4 * c) + v][lane] = t;
      }
    __syncthreads();
    const int a = 4 * c + w;
    if (a < NU) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = 4 * w + v;
        const floatx4 o = ((red[0][i][lane] + red[1][i][lane]) + red[2][i][lane]) + red[3][i][lane];
        int m = 0;
        // U::row with a wave-uniform block index
#pragma unroll
        for (int aa = 4 * c; aa < 4 * c + 4 && aa < NU; ++aa)
          if (aa == a) m = U::row(aa, 4 * gq + v);
        if (m >= M) continue;
        float* orow = out + (int64_t)m * p.ld0 + n0;
        if constexpr (X::NB == 4 && X::B2 == 64) {
          // one 16-byte segment: inputs 4 r .. 4 r + 3
          if (4 * r < N - n0) *reinterpret_cast<floatx4*>(orow + 4 * r) = o;
        } else {
#pragma unroll
          for (int b = 0; b < NX; ++b) {
            const int n = X::row(b, r);
            if (n < N - n0) orow[n] = o[b];
          }
        }
      }
    }
  }
  if (do_bias && tid < M)
    p.pbias[(int64_t)piece * M + tid] =
        ((bred[0][tid] + bred[1][tid]) + bred[2][tid]) + bred[3][tid];
}

// the tile's input side: a whole tile of 64 inputs, or the last tile's
// ceil(rest / 16) blocks
template <class U>
__device__ __forceinline__ void skinny_tile_x(const GemmParamsT<float>& p, int piece, int tile,
                                              int nx, floatx4 (*red)[16][64],
                                              float (*bred)[SKINNY_MAX_UNITS]) {
  switch (nx) {
    case 1: skinny_tile<U, SkSide<0, 0, 1>>(p, piece, tile, red, bred); break;
    case 2: skinny_tile<U, SkSide<0, 1, 0>>(p, piece, tile, red, bred); break;
    case 3: skinny_tile<U, SkSide<0, 1, 1>>(p, piece, tile, red, bred); break;
    default: skinny_tile<U, SkSide<1, 0, 0>>(p, piece, tile, red, bred); break;
  }
}

__global__ void __launch_bounds__(SK_NT, 2) skinny_dw_kernel(const SkinnyGroup g) {
  // the four waves' accumulators of four unit blocks, [wave][slot][lane],
  // and the bias sums
  __shared__ floatx4 red[4][16][64];
  __shared__ float bred[4][SKINNY_MAX_UNITS];

  const int b = blockIdx.x;
  int q = 0;
#pragma unroll
  for (int i = 1; i < GEMM_GROUP_MAX; ++i) q += (i < g.n && b >= g.start[i]);
  const GemmParamsT<float>& p = g.p[q];
  const int ntile = (p.N + SK_TN - 1) / SK_TN;
  const int r0 = b - g.start[q];
  const int slot = r0 >> 3;
  const int piece = (r0 & 7) + 8 * (slot / ntile);
  const int tile = slot % ntile;
  if (piece >= g.npieces[q]) return;
  const int rest = p.N - tile * SK_TN;
  const int nx = rest >= SK_TN ? 4 : (rest + 15) >> 4;
  switch ((p.M + 15) >> 4) {
    case 1: skinny_tile_x<SkSide<0, 0, 1>>(p, piece, tile, nx, red, bred); break;
    case 2: skinny_tile_x<SkSide<0, 1, 0>>(p, piece, tile, nx, red, bred); break;
    case 3: skinny_tile_x<SkSide<0, 1, 1>>(p, piece, tile, nx, red, bred); break;
    case 4: skinny_tile_x<SkSide<1, 0, 0>>(p, piece, tile, nx, red, bred); break;
    case 5: skinny_tile_x<SkSide<1, 0, 1>>(p, piece, tile, nx, red, bred); break;
    case 6: skinny_tile_x<SkSide<1, 1, 0>>(p, piece, tile, nx, red, bred); break;
    case 7: skinny_tile_x<SkSide<1, 1, 1>>(p, piece, tile, nx, red, bred); break;
    default: skinny_tile_x<SkSide<2, 0, 0>>(p, piece, tile, nx, red, bred); break;
  }
}

// ---------------------------------------------------------------------------
// fp64 tendency pieces: the same design on v_mfma_f64_16x16x4f64.  A 16-byte
// load holds two doubles, so the wide segments are 32 rows (row 2 r + e of a
// segment is row r of its block e) and the last 16 rows take 8-byte loads;
// input tiles are 32 wide (two blocks).  The accumulator layout differs from
// fp32: register v of lane (r, g) is row 4 v + g of the block.
// ---------------------------------------------------------------------------
typedef double doublex2 __attribute__((ext_vector_type(2)));
typedef double doublex4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ doublex2 sk_load_d2(__amdgpu_buffer_rsrc_t rs, unsigned off) {
  return __builtin_bit_cast(doublex2, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
}
__device__ __forceinline__ double sk_load_d1(__amdgpu_buffer_rsrc_t rs, unsigned off) {
  return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0));
}

// One side of an fp64 tile: S2 segments of 32 rows (16-byte loads), then S1
// <= 1 segment of 16 rows (8-byte loads).
template <int S2, int S1>
struct SkSide64 {
  static constexpr int NB = 2 * S2 + S1;
  static constexpr int B1 = 32 * S2;
  __device__ static int row(int b, int r) {
    if (b < 2 * S2) return 32 * (b >> 1) + 2 * r + (b & 1);
    return B1 + r;
  }
  struct Regs {
    doublex2 v2[S2 > 0 ? S2 : 1];
    double v1;
  };
  __device__ static void load(Regs& g, __amdgpu_buffer_rsrc_t rs, unsigned base, int r, int lim,
                              bool ok) {
#pragma unroll
    for (int i = 0; i < S2; ++i) {
      const int e = 32 * i + 2 * r;
      g.v2[i] = sk_load_d2(rs, ok && e < lim ? base + 8u * (unsigned)e : SK_OOB);
    }
    if constexpr (S1 > 0) {
      const int e = B1 + r;
      g.v1 = sk_load_d1(rs, ok && e < lim ? base + 8u * (unsigned)e : SK_OOB);
    }
  }
  __device__ static double at(const Regs& g, int b) {
    if (b < 2 * S2) return g.v2[b >> 1][b & 1];
    return g.v1;
  }
};

constexpr int SK64_TN = SKINNY_TILE_F64;

template <class U, class X>
__device__ __forceinline__ void skinny_tile64(const GemmParamsT<double>& p, int piece, int tile,
                                              doublex2 (*red)[16][64],
                                              double (*bred)[SKINNY_MAX_UNITS]) {
  constexpr int NU = U::NB, NX = X::NB;
  static_assert(NX <= 2, "two input blocks per tile");
  const int M = p.M, N = p.N;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15, gq = lane >> 4;
  const int n0 = tile * SK64_TN;
  const bool do_bias = tile == 0;

  const int shard = piece / p.nsub, sub = piece % p.nsub;
  const int sb = shard * p.shard_len;
  const int kbeg = sb + sub * p.sub_len;
  const int kend = min(kbeg + p.sub_len, sb + p.shard_len);
  const int nks = kend > kbeg ? (kend - kbeg + 3) >> 2 : 0;
  const int qk = (nks + 3) >> 2;
  const int j0 = min(nks, w * qk), j1 = min(nks, j0 + qk);
  const int lda = (int)p.lda, ldb = (int)p.ldb;
  const unsigned dbase = 8u * (unsigned)(gq * lda), xbase = 8u * (unsigned)(gq * ldb + n0);

  doublex4 acc[NU][NX];
#pragma unroll
  for (int a = 0; a < NU; ++a)
#pragma unroll
    for (int b = 0; b < NX; ++b) acc[a][b] = doublex4{0.0, 0.0, 0.0, 0.0};
  double bsum[NU];
#pragma unroll
  for (int a = 0; a < NU; ++a) bsum[a] = 0.0;

  struct Step {
    typename U::Regs d;
    typename X::Regs x;
  };
  auto load = [&](Step& st, int j) {
    const int s0 = kbeg + 4 * j;
    const bool ok = j < j1 && s0 + gq < kend;
    U::load(st.d, sk_rsrc(reinterpret_cast<const float*>(p.A + (int64_t)s0 * lda)), dbase, r, M, ok);
    X::load(st.x, sk_rsrc(reinterpret_cast<const float*>(p.B + (int64_t)s0 * ldb)), xbase, r,
            N - n0, ok);
  };
  auto step = [&](const Step& st) {
#pragma unroll
    for (int a = 0; a < NU; ++a)
#pragma unroll
      for (int b = 0; b < NX; ++b)
        acc[a][b] = __builtin_amdgcn_mfma_f64_16x16x4f64(U::at(st.d, a), X::at(st.x, b), acc[a][b],
                                                         0, 0, 0);
    if (do_bias) {
#pragma unroll
      for (int a = 0; a < NU; ++a) bsum[a] += U::at(st.d, a);
    }
  };

  constexpr int PD = SKINNY_PD;
  Step st[PD];
#pragma unroll
  for (int d = 0; d < PD; ++d) load(st[d], j0 + d);
  int j = j0;
  for (; j + PD <= j1; j += PD) {
#pragma unroll
    for (int d = 0; d < PD; ++d) {
      step(st[d]);
      load(st[d], j + d + PD);
    }
  }
#pragma unroll
  for (int d = 0; d < PD - 1; ++d)
    if (j + d < j1) step(st[d]);

  if (do_bias) {
#pragma unroll
    for (int a = 0; a < NU; ++a) {
      double t = bsum[a];
      t += __shfl_xor(t, 16);
      t += __shfl_xor(t, 32);
      if (gq == 0) bred[w][U::row(a, r)] = t;
    }
  }

  // Unit blocks 4 c .. 4 c + 3 at a time, as in fp32; accumulator register
  // v of lane (r, gq) is row 4 v + gq of the block, column r.
  double* out = p.partial + (int64_t)piece * p.pstride;
#pragma unroll
  for (int c = 0; c < (NU + 3) / 4; ++c) {
    if (c > 0) __syncthreads();
#pragma unroll
    for (int a = 4 * c; a < 4 * c + 4 && a < NU; ++a)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        doublex2 t = doublex2{0.0, 0.0};
#pragma unroll
        for (int b = 0; b < NX; ++b) t[b] = acc[a][b][v];
        red[w][4 * (a - 4 * c) + v][lane] = t;
      }
    __syncthreads();
    const int a = 4 * c + w;
    if (a < NU) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = 4 * w + v;
        const doublex2 o = ((red[0][i][lane] + red[1][i][lane]) + red[2][i][lane]) + red[3][i][lane];
        int m = 0;
#pragma unroll
        for (int aa = 4 * c; aa < 4 * c + 4 && aa < NU; ++aa)
          if (aa == a) m = U::row(aa, 4 * v + gq);
        if (m >= M) continue;
        double* orow = out + (int64_t)m * p.ld0 + n0;
#pragma unroll
        for (int b = 0; b < NX; ++b) {
          const int n = X::row(b, r);
          if (n < N - n0) orow[n] = o[b];
        }
      }
    }
  }
  if (do_bias && tid < M)
    p.pbias[(int64_t)piece * M + tid] =
        ((bred[0][tid] + bred[1][tid]) + bred[2][tid]) + bred[3][tid];
}

template <class U>
__device__ __forceinline__ void skinny_tile64_x(const GemmParamsT<double>& p, int piece, int tile,
                                                int nx, doublex2 (*red)[16][64],
                                                double (*bred)[SKINNY_MAX_UNITS]) {
  if (nx == 1)
    skinny_tile64<U, SkSide64<0, 1>>(p, piece, tile, red, bred);
  else
    skinny_tile64<U, SkSide64<1, 0>>(p, piece, tile, red, bred);
}

__global__ void __launch_bounds__(SK_NT, 2) skinny_dw64_kernel(const SkinnyGroup64 g) {
  __shared__ doublex2 red[4][16][64];
  __shared__ double bred[4][SKINNY_MAX_UNITS];

  const int b = blockIdx.x;
  int q = 0;
#pragma unroll
  for (int i = 1; i < GEMM_GROUP_MAX; ++i) q += (i < g.n && b >= g.start[i]);
  const GemmParamsT<double>& p = g.p[q];
  const int ntile = (p.N + SK64_TN - 1) / SK64_TN;
  const int r0 = b - g.start[q];
  const int slot = r0 >> 3;
  const int piece = (r0 & 7) + 8 * (slot / ntile);
  const int tile = slot % ntile;
  if (piece >= g.npieces[q]) return;
  const int rest = p.N - tile * SK64_TN;
  const int nx = rest >= SK64_TN ? 2 : (rest + 15) >> 4;
  switch ((p.M + 15) >> 4) {
    case 1: skinny_tile64_x<SkSide64<0, 1>>(p, piece, tile, nx, red, bred); break;
    case 2: skinny_tile64_x<SkSide64<1, 0>>(p, piece, tile, nx, red, bred); break;
    case 3: skinny_tile64_x<SkSide64<1, 1>>(p, piece, tile, nx, red, bred); break;
    case 4: skinny_tile64_x<SkSide64<2, 0>>(p, piece, tile, nx, red, bred); break;
    case 5: skinny_tile64_x<SkSide64<2, 1>>(p, piece, tile, nx, red, bred); break;
    case 6: skinny_tile64_x<SkSide64<3, 0>>(p, piece, tile, nx, red, bred); break;
    case 7: skinny_tile64_x<SkSide64<3, 1>>(p, piece, tile, nx, red, bred); break;
    default: skinny_tile64_x<SkSide64<4, 0>>(p, piece, tile, nx, red, bred); break;
  }
}

// ---------------------------------------------------------------------------
// Forward pieces of a layer of at most SKINNY_MAX_UNITS units (section 3.2:
// z[s][u] = sum over inputs n of x[s][n] W[u][n], over one piece of the
// input range).  The k index is contiguous in both operands, so lane (r, g)
// takes inputs k0 + 4 g .. + 3 of a row in one 16-byte access and uses them
// in the 4 products of a k-group of 16 inputs.
//
// A workgroup of 8 waves owns one piece and 8 blocks of 16 samples.  It
// copies the piece's slice of W (every unit, the piece's inputs) into LDS,
// at a row pitch of 4 (odd) floats so that the 16 rows of a fragment read
// fall on distinct banks, in two parts: the first SKINNY_FWD_PD k-groups
// (when the piece has at least twice as many), then the rest, whose loads
// are in flight while the first part's products run.  After each part's
// barrier every wave runs its own sample block: the sample rows come from
// global memory, SKINNY_FWD_PD k-groups ahead, the unit rows from LDS.
// ---------------------------------------------------------------------------
constexpr int SKF_NT = 512;    // 8 waves
constexpr int SKF_BATCH = 8;   // 16-byte copy loads per thread in one round

// the 16-byte chunks of one round of the copy: values and LDS offsets
struct SkfChunks {
  floatx4 v[SKF_BATCH];
  int at[SKF_BATCH];
};

template <int NUB, class Stage>
__device__ __forceinline__ void fwd_skinny_tile(const GemmParamsT<float>& p, int sblk, int piece,
                                                const float* ws, int pk, Stage& stage) {
  const int lane = threadIdx.x & 63;
  const int r = lane & 15, gq = lane >> 4;
  const int M = p.M, N = p.N;
  const int s0 = 16 * sblk;
  const int kbeg = piece * p.sub_len;
  const int kend = min(kbeg + p.sub_len, p.K);
  const int ngr = kend > kbeg ? (kend - kbeg + 15) >> 4 : 0;   // k-groups of 16 inputs
  const bool xok = s0 + r < M;
  const __amdgpu_buffer_rsrc_t ra = sk_rsrc(p.A + (int64_t)s0 * p.lda);
  const int lda = (int)p.lda;

  floatx4 acc[NUB];
#pragma unroll
  for (int u = 0; u < NUB; ++u) acc[u] = floatx4{0.f, 0.f, 0.f, 0.f};
  // k-group t: inputs kbeg + 16 t + 4 gq .. + 3 (whole vectors: the pieces
  // start on multiples of 16 and the row length is a multiple of 4)
  auto load = [&](int t) {
    const int k = kbeg + 16 * t + 4 * gq;
    return sk_load(ra, k < kend && xok ? 4u * (unsigned)(r * lda + k) : SK_OOB);
  };
  const float* wl = ws + r * pk + 4 * gq;
  auto step = [&](const floatx4& xv, int t) {
    floatx4 wv[NUB];
#pragma unroll
    for (int u = 0; u < NUB; ++u)
      wv[u] = *reinterpret_cast<const floatx4*>(wl + 16 * u * pk + 16 * t);
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int u = 0; u < NUB; ++u)
        acc[u] = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[tt], wv[u][tt], acc[u], 0, 0, 0);
  };
  constexpr int PD = SKINNY_FWD_PD;
  const bool has_rows = s0 < M;
  // the copy's split: k-groups [0, hs) first, 4 hs chunk columns
  const int hs = ngr >= 2 * PD ? PD : 0;
  // the first part's loads (from the L2) issue before the sample rows' (from
  // memory), so that they are not queued behind them; the second part's
  // first round follows the sample rows
  SkfChunks g1, g2;
  stage.issue(g1, 0, 4 * hs, 0);
  floatx4 xv[PD];
#pragma unroll
  for (int d = 0; d < PD; ++d) xv[d] = load(d);
  stage.issue(g2, 4 * hs, 4 * ngr, 0);
  stage.store(g1);
  stage.copy(0, 4 * hs, 1);
  __syncthreads();
  int t = 0;
  if (has_rows && hs == PD) {
#pragma unroll
    for (int d = 0; d < PD; ++d) {
      step(xv[d], d);
      xv[d] = load(d + PD);
    }
    t = PD;
  }
  stage.store(g2);
  stage.copy(4 * hs, 4 * ngr, 1);
  __syncthreads();
  if (!has_rows) return;
  for (; t + PD <= ngr; t += PD) {
#pragma unroll
    for (int d = 0; d < PD; ++d) {
      step(xv[d], t + d);
      xv[d] = load(t + d + PD);
    }
  }
#pragma unroll
  for (int d = 0; d < PD - 1; ++d)
    if (t + d < ngr) step(xv[d], t + d);

  // accumulator register v of lane (r, gq): sample s0 + 4 gq + v, unit 16 u + r
  float* out = p.partial + (int64_t)piece * p.pstride;
#pragma unroll
  for (int u = 0; u < NUB; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int m = s0 + 4 * gq + v;
      if (m < M && 16 * u + r < N) out[(int64_t)m * p.ld0 + 16 * u + r] = acc[u][v];
    }
}

// The copy of a piece's slice of W: row u, inputs kbeg .. kend - 1 at
// ws[u * pk + ..], zeros up to the end of the last k-group (their products
// meet the zeros that the sample loads past kend return).  A part of it is
// the chunk columns [c0, c1) (4 floats each) of every row: chunk i of the
// part is row i / w, column c0 + i % w with w = c1 - c0, the quotient a
// multiply-high by floor(2^32 / w) + 1, exact while i w < 2^32 (the slice
// fits in LDS, so both stay below 2^14).  Chunks past the part go to the
// spare 16 bytes after the slice's rows, so no store is tied to a branch.
struct SkfStage {
  const GemmParamsT<float>& p;
  float* ws;
  int pk, kbeg, kend, spare, ldb;
  __amdgpu_buffer_rsrc_t rb;

  __device__ SkfStage(const GemmParamsT<float>& p_, float* ws_, int pk_, int piece) : p(p_), ws(ws_), pk(pk_) {
    kbeg = piece * p.sub_len;
    kend = min(kbeg + p.sub_len, p.K);
    spare = 16 * ((p.N + 15) >> 4) * pk;
    ldb = (int)p.ldb;
    rb = sk_rsrc(p.B + kbeg);
  }
  __device__ int rounds(int c0, int c1) const {
    const int total = p.N * (c1 - c0);
    return total > 0 ? (total + SKF_BATCH * SKF_NT - 1) / (SKF_BATCH * SKF_NT) : 0;
  }
  // round q of the part's loads
  __device__ void issue(SkfChunks& g, int c0, int c1, int q) const {
    const int w = c1 - c0, total = p.N * w;
    const unsigned mq = w > 0 ? 0xffffffffu / (unsigned)w + 1u : 0u;
#pragma unroll
    for (int j = 0; j < SKF_BATCH; ++j) {
      const int i = (q * SKF_BATCH + j) * SKF_NT + (int)threadIdx.x;
      const int u = (int)__umulhi((unsigned)i, mq), c = c0 + i - u * w;
      const bool in = i < total;
      g.at[j] = in ? u * pk + 4 * c : spare;
      g.v[j] = sk_load(rb, in && kbeg + 4 * c < kend ? 4u * (unsigned)(u * ldb + 4 * c) : SK_OOB);
    }
  }
  __device__ void store(const SkfChunks& g) const {
#pragma unroll
    for (int j = 0; j < SKF_BATCH; ++j) *reinterpret_cast<floatx4*>(ws + g.at[j]) = g.v[j];
  }
  // rounds from q0 on, each loaded and stored in turn
  __device__ void copy(int c0, int c1, int q0) const {
    const int nq = rounds(c0, c1);
    for (int q = q0; q < nq; ++q) {
      SkfChunks g;
      issue(g, c0, c1, q);
      store(g);
    }
  }
};

__global__ void __launch_bounds__(SKF_NT) fwd_skinny_kernel(const GemmParamsT<float> p, int pk) {
  extern __shared__ floatx4 ws4[];
  float* ws = reinterpret_cast<float*>(ws4);
  // workgroup b: piece b % nsub, sample blocks 8 (b / nsub) .. + 7
  const int piece = blockIdx.x % p.nsub;
  const int sblk = 8 * (blockIdx.x / p.nsub) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  SkfStage stage(p, ws, pk, piece);
  switch ((p.N + 15) >> 4) {
    case 1: fwd_skinny_tile<1>(p, sblk, piece, ws, pk, stage); break;
    case 2: fwd_skinny_tile<2>(p, sblk, piece, ws, pk, stage); break;
    case 3: fwd_skinny_tile<3>(p, sblk, piece, ws, pk, stage); break;
    case 4: fwd_skinny_tile<4>(p, sblk, piece, ws, pk, stage); break;
    case 5: fwd_skinny_tile<5>(p, sblk, piece, ws, pk, stage); break;
    case 6: fwd_skinny_tile<6>(p, sblk, piece, ws, pk, stage); break;
    case 7: fwd_skinny_tile<7>(p, sblk, piece, ws, pk, stage); break;
    default: fwd_skinny_tile<8>(p, sblk, piece, ws, pk, stage); break;
  }
}

}  // namespace

hipError_t launch_dw_skinny_group(SkinnyGroup g, hipStream_t s) {
  if (g.n < 1 || g.n > GEMM_GROUP_MAX) return hipErrorInvalidValue;
  g.start[0] = 0;
  for (int q = 0; q < g.n; ++q) {
    const GemmParamsT<float>& p = g.p[q];
    if (p.M <= 0 || p.M > SKINNY_MAX_UNITS || p.N <= 0 || p.K < 0 || g.npieces[q] <= 0)
      return hipErrorInvalidValue;
    if (p.nsub <= 0 || g.npieces[q] % p.nsub != 0) return hipErrorInvalidValue;
    // 16-byte loads of rows and stores of tendency rows: pitches of whole
    // vectors, 16-byte aligned bases
    if (p.lda % 4 != 0 || p.ldb % 4 != 0 || p.ld0 % 4 != 0 || p.pstride % 4 != 0 ||
        p.lda < 4 * ((p.M + 3) / 4) || p.ldb < 4 * ((p.N + 3) / 4) || p.ld0 < 4 * ((p.N + 3) / 4))
      return hipErrorInvalidValue;
    if ((reinterpret_cast<uintptr_t>(p.A) & 15) != 0 || (reinterpret_cast<uintptr_t>(p.B) & 15) != 0 ||
        (reinterpret_cast<uintptr_t>(p.partial) & 15) != 0)
      return hipErrorInvalidValue;
    // a k-step's offsets are 32-bit, within 4 rows of its first row
    const int64_t ld = p.lda > p.ldb ? p.lda : p.ldb;
    if ((int64_t)4 * ld * 4 >= (int64_t)SK_OOB) return hipErrorInvalidValue;
    const int ntile = (p.N + SK_TN - 1) / SK_TN;
    g.start[q + 1] = g.start[q] + 8 * ((g.npieces[q] + 7) / 8) * ntile;
  }
  for (int q = g.n + 1; q <= GEMM_GROUP_MAX; ++q) g.start[q] = g.start[g.n];
  if (g.start[g.n] <= 0) return hipErrorInvalidValue;
  return launch_k(skinny_dw_kernel, dim3((unsigned)g.start[g.n]), dim3(SK_NT), 0, s, g);
}

int fwd_skinny_pitch(int sub_len) {
  // whole k-groups, then a multiple of 4 floats whose quarter is odd: rows
  // r = 0..15 of a 16-byte fragment read start in 16 distinct groups of 4
  // banks
  const int q = 4 * ((sub_len + 15) / 16);
  return 4 * (q % 2 == 1 ? q : q + 1);
}

int64_t fwd_skinny_lds_bytes(int N, int sub_len) {
  // the slice's rows, padded to 16 units, and a spare 16-byte slot
  return (int64_t)16 * ((N + 15) / 16) * fwd_skinny_pitch(sub_len) * 4 + 16;
}

hipError_t launch_dw_skinny_group64(SkinnyGroup64 g, hipStream_t s) {
  if (g.n < 1 || g.n > GEMM_GROUP_MAX) return hipErrorInvalidValue;
  g.start[0] = 0;
  for (int q = 0; q < g.n; ++q) {
    const GemmParamsT<double>& p = g.p[q];
    if (p.M <= 0 || p.M > SKINNY_MAX_UNITS || p.N <= 0 || p.K < 0 || g.npieces[q] <= 0)
      return hipErrorInvalidValue;
    if (p.nsub <= 0 || g.npieces[q] % p.nsub != 0) return hipErrorInvalidValue;
    // 16-byte loads of two doubles: even pitches, rows 16-byte aligned
    if (p.lda % 2 != 0 || p.ldb % 2 != 0 || p.lda < 2 * ((p.M + 1) / 2) ||
        p.ldb < 2 * ((p.N + 1) / 2) || p.ld0 < p.N)
      return hipErrorInvalidValue;
    if ((reinterpret_cast<uintptr_t>(p.A) & 15) != 0 || (reinterpret_cast<uintptr_t>(p.B) & 15) != 0)
      return hipErrorInvalidValue;
    const int64_t ld = p.lda > p.ldb ? p.lda : p.ldb;
    if ((int64_t)4 * ld * 8 >= (int64_t)SK_OOB) return hipErrorInvalidValue;
    const int ntile = (p.N + SK64_TN - 1) / SK64_TN;
    g.start[q + 1] = g.start[q] + 8 * ((g.npieces[q] + 7) / 8) * ntile;
  }
  for (int q = g.n + 1; q <= GEMM_GROUP_MAX; ++q) g.start[q] = g.start[g.n];
  if (g.start[g.n] <= 0) return hipErrorInvalidValue;
  return launch_k(skinny_dw64_kernel, dim3((unsigned)g.start[g.n]), dim3(SK_NT), 0, s, g);
}

hipError_t launch_fwd_skinny(const GemmParamsT<float>& p, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0 || p.N > SKINNY_MAX_UNITS || p.K <= 0 || p.nsub <= 0)
    return hipErrorInvalidValue;
  // pieces after the first start on whole k-groups; 16-byte row loads
  if (p.sub_len <= 0 || (p.nsub > 1 && p.sub_len % 16 != 0) || (int64_t)p.nsub * p.sub_len < p.K ||
      (int64_t)(p.nsub - 1) * p.sub_len >= p.K)
    return hipErrorInvalidValue;
  if (p.K % 4 != 0 || p.lda % 4 != 0 || p.ldb % 4 != 0 || p.lda < p.K || p.ldb < p.K ||
      p.ld0 < p.N)
    return hipErrorInvalidValue;
  if ((reinterpret_cast<uintptr_t>(p.A) & 15) != 0 || (reinterpret_cast<uintptr_t>(p.B) & 15) != 0)
    return hipErrorInvalidValue;
  // 32-bit offsets: 16 rows of A past the block's first row, every row of B
  if ((int64_t)16 * p.lda * 4 >= (int64_t)SK_OOB || (int64_t)p.N * p.ldb * 4 >= (int64_t)SK_OOB)
    return hipErrorInvalidValue;
  const int64_t lds = fwd_skinny_lds_bytes(p.N, p.sub_len);
  if (lds > SKINNY_FWD_LDS) return hipErrorInvalidValue;
  const int64_t groups = ((int64_t)p.M + 127) / 128;
  if (groups * p.nsub > 0x7fffffff) return hipErrorInvalidValue;
  // the kernel may use more than the default dynamic LDS: allowed once per
  // device (any thread may get there first; the call is idempotent)
  constexpr int kDevices = 64;
  static std::atomic<bool> attr_set[kDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kDevices || !attr_set[dev].load(std::memory_order_acquire)) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(fwd_skinny_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, SKINNY_FWD_LDS);
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < kDevices) attr_set[dev].store(true, std::memory_order_release);
  }
  return launch_k(fwd_skinny_kernel, dim3((unsigned)(groups * p.nsub)), dim3(SKF_NT),
                  (unsigned)lds, s, p, fwd_skinny_pitch(p.sub_len));
}

}  // namespace nf
