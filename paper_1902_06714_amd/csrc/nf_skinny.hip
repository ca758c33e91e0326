// Tendency pieces (section 3.3: dC/dW_l = delta_l^T a_{l-1}, dC/db_l = the
// column sums of delta_l, each over one piece of the batch) of fp32 layers
// with at most SKINNY_MAX_UNITS units, e.g. the 100-unit layers of a
// 784-100-100-10 network.
//
// Both operands are sample-major (delta_l[s][u], a_{l-1}[s][n]) and the sum
// runs over samples, so a 16-byte load gives a lane 4 consecutive units (or
// inputs) of one sample.  The kernel takes them straight from global memory
// into matrix-core operands, with no LDS staging and no barrier in the loop:
// in a 16x16x4 product lane (r, g) supplies row r of A and column r of B at
// input index g, so the 4 values of a lane's vector go to 4 different
// products.  Unit 4 r + e of a group of 64 is row r of unit block e, input
// 4 r + e' of a tile of 64 is column r of input block e', and input index g
// is sample 4 j + g of k-step j.  A wave holds the 4 x 4 blocks of each
// group of 64 units (one or two groups) against one tile of 64 inputs and
// per k-step of 4 samples issues one 16-byte load per unit group and one for
// the inputs (each a 4 rows x 256 bytes pattern) for 16 products per unit
// group.  SKINNY_PD k-steps of loads are in flight.
//
// A workgroup of 4 waves owns one (piece, input tile): wave w takes the w-th
// quarter of the piece's k-steps, and the four partial sums are added
// through LDS in wave order at the end, one unit group at a time.  A tile-0
// workgroup also sums the delta columns (the bias tendency): each lane over
// its samples, then over the 4 lanes of a unit, then over the waves.
//
// Workgroups go round robin over the 8 XCDs (workgroup b runs on XCD b mod
// 8).  XCD x takes pieces x, x + 8, ... of a layer, each with all of its
// input tiles one after another, so a piece's delta rows are fetched into
// that XCD's L2 once.
//
// The per-piece sums land in the same [piece][M][ld0] + [piece][M] layout as
// the general tendency pieces, and fold_sgd_kernel folds them in piece order.
#include "nf_internal.h"

namespace nf {

typedef float floatx4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int SK_NT = 256;                 // 4 waves
constexpr int SK_TN = 64;                  // inputs per tile
constexpr int SK_TU = 64;                  // units per group
constexpr unsigned SK_OOB = 0x7ffffff0u;   // buffer length: offsets past it read 0
static_assert(SKINNY_MAX_UNITS <= 2 * SK_TU, "two unit groups at most");

__device__ __forceinline__ __amdgpu_buffer_rsrc_t sk_rsrc(const float* base) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, (int)SK_OOB, 0x00020000);
}

__device__ __forceinline__ floatx4 sk_load(__amdgpu_buffer_rsrc_t rs, unsigned off) {
  return __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
}

// One workgroup's (piece, input tile) with NG groups of 64 units (the
// layer's units rounded up).
template <int NG>
__device__ __forceinline__ void skinny_tile(const GemmParamsT<float>& p, int piece, int tile,
                                            floatx4 (*red)[16][64], float (*bred)[SKINNY_MAX_UNITS]) {
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

  // this lane's columns: units 64 c + 4 r .. + 3 of delta (group c), inputs
  // n0 + 4 r .. + 3
  bool dok[NG];
  unsigned doff[NG];
#pragma unroll
  for (int c = 0; c < NG; ++c) {
    dok[c] = SK_TU * c + 4 * r < M;
    doff[c] = 4u * (unsigned)(gq * (int)p.lda + SK_TU * c + 4 * r);
  }
  const bool xok = n0 + 4 * r < N;
  const int lda = (int)p.lda, ldb = (int)p.ldb;
  const unsigned xoff = 4u * (unsigned)(gq * ldb + n0 + 4 * r);

  floatx4 acc[NG][4][4];
#pragma unroll
  for (int c = 0; c < NG; ++c)
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int f = 0; f < 4; ++f) acc[c][e][f] = floatx4{0.f, 0.f, 0.f, 0.f};
  floatx4 bsum[NG];
#pragma unroll
  for (int c = 0; c < NG; ++c) bsum[c] = floatx4{0.f, 0.f, 0.f, 0.f};

  struct Step {
    floatx4 d[NG], x;
  };
  // k-step j: samples kbeg + 4 j + gq; past j1 or kend the loads read zeros
  auto load = [&](Step& st, int j) {
    const int s0 = kbeg + 4 * j;
    const bool ok = j < j1 && s0 + gq < kend;
    const __amdgpu_buffer_rsrc_t ra = sk_rsrc(p.A + (int64_t)s0 * lda);
#pragma unroll
    for (int c = 0; c < NG; ++c) st.d[c] = sk_load(ra, ok && dok[c] ? doff[c] : SK_OOB);
    st.x = sk_load(sk_rsrc(p.B + (int64_t)s0 * ldb), ok && xok ? xoff : SK_OOB);
  };
  auto step = [&](const Step& st) {
#pragma unroll
    for (int c = 0; c < NG; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int f = 0; f < 4; ++f)
          acc[c][e][f] = __builtin_amdgcn_mfma_f32_16x16x4f32(st.d[c][e], st.x[f], acc[c][e][f], 0, 0, 0);
    if (do_bias) {
#pragma unroll
      for (int c = 0; c < NG; ++c) bsum[c] += st.d[c];
    }
  };

  // SKINNY_PD k-steps of loads in flight; whole groups load unconditionally
  // (past the wave's range the loads read zeros), so each wait is for
  // exactly the k-step needed
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
    // lanes r, r + 16, r + 32, r + 48 hold the same units
#pragma unroll
    for (int c = 0; c < NG; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float s = bsum[c][e];
        s += __shfl_xor(s, 16);
        s += __shfl_xor(s, 32);
        if (gq == 0) bred[w][SK_TU * c + 4 * r + e] = s;
      }
  }

  // One unit group at a time: the 4 input blocks f of a lane's (unit block
  // e, accumulator row v) go to LDS as one vector, slot 4 e + v; wave w then
  // sums slots 4 w .. 4 w + 3 over the waves in wave order and stores rows
  // 64 c + 16 gq + 4 v + w, inputs n0 + 4 r .. + 3.
  float* out = p.partial + (int64_t)piece * p.pstride;
#pragma unroll
  for (int c = 0; c < NG; ++c) {
    if (c > 0) __syncthreads();   // the previous group's sums are read
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        red[w][4 * e + v][lane] =
            floatx4{acc[c][e][0][v], acc[c][e][1][v], acc[c][e][2][v], acc[c][e][3][v]};
    __syncthreads();
    if (xok) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = SK_TU * c + 16 * gq + 4 * v + w;
        const int i = 4 * w + v;
        const floatx4 o = ((red[0][i][lane] + red[1][i][lane]) + red[2][i][lane]) + red[3][i][lane];
        if (m < M) *reinterpret_cast<floatx4*>(out + (int64_t)m * p.ld0 + n0 + 4 * r) = o;
      }
    }
  }
  if (do_bias && tid < M)
    p.pbias[(int64_t)piece * M + tid] =
        ((bred[0][tid] + bred[1][tid]) + bred[2][tid]) + bred[3][tid];
}

__global__ void __launch_bounds__(SK_NT, 2) skinny_dw_kernel(const SkinnyGroup g) {
  // the four waves' accumulators of one unit group, [wave][value][lane],
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
  if (p.M > SK_TU)
    skinny_tile<2>(p, piece, tile, red, bred);
  else
    skinny_tile<1>(p, piece, tile, red, bred);
}

// ---------------------------------------------------------------------------
// Forward pieces of a layer of at most SKINNY_MAX_UNITS units (section 3.2:
// z[s][u] = sum over inputs n of x[s][n] W[u][n], over one piece of the
// input range).  The k index is contiguous in both operands, so lane (r, g)
// takes inputs k0 + 4 g .. + 3 of a row in one 16-byte access and uses them
// in the 4 products of a k-group of 16 inputs.
//
// A workgroup of 8 waves owns one piece and 8 blocks of 16 samples.  It
// first copies the piece's slice of W (every unit, the piece's inputs) into
// LDS, at a row pitch of 4 (odd) floats so that the 16 rows of a fragment
// read fall on distinct banks; after that one barrier each wave runs its
// own sample block: the sample rows come from global memory, SKINNY_FWD_PD
// k-groups ahead, the unit rows from LDS.
// ---------------------------------------------------------------------------
constexpr int SKF_NT = 512;   // 8 waves

template <int NUB>
__device__ __forceinline__ void fwd_skinny_tile(const GemmParamsT<float>& p, int sblk, int piece,
                                                const float* ws, int pk) {
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
  floatx4 xv[PD];
#pragma unroll
  for (int d = 0; d < PD; ++d) xv[d] = load(d);
  int t = 0;
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

__global__ void __launch_bounds__(SKF_NT) fwd_skinny_kernel(const GemmParamsT<float> p, int pk) {
  extern __shared__ floatx4 ws4[];
  float* ws = reinterpret_cast<float*>(ws4);
  // workgroup b: piece b % nsub, sample blocks 8 (b / nsub) .. + 7
  const int piece = blockIdx.x % p.nsub;
  const int sblk = 8 * (blockIdx.x / p.nsub) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

  // the piece's slice of W: row u, inputs kbeg .. kend - 1 at ws[u * pk + ..],
  // zeros up to the end of the last k-group (their products meet the zeros
  // that the sample loads past kend return)
  const int kbeg = piece * p.sub_len;
  const int kend = min(kbeg + p.sub_len, p.K);
  const int len4 = 4 * ((kend - kbeg + 15) >> 4);
  const int total = p.N * len4;
  const __amdgpu_buffer_rsrc_t rb = sk_rsrc(p.B + kbeg);
  const int ldb = (int)p.ldb;
  constexpr int BATCH = 16;   // 16-byte loads per thread in flight at once
  for (int i0 = 0; i0 < total; i0 += BATCH * SKF_NT) {
    floatx4 v[BATCH];
    int at[BATCH];
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int i = i0 + j * SKF_NT + (int)threadIdx.x;
      const int u = i / len4, c = i - u * len4;
      at[j] = i < total ? u * pk + 4 * c : -1;
      v[j] = sk_load(rb, i < total && kbeg + 4 * c < kend ? 4u * (unsigned)(u * ldb + 4 * c) : SK_OOB);
    }
#pragma unroll
    for (int j = 0; j < BATCH; ++j)
      if (at[j] >= 0) *reinterpret_cast<floatx4*>(ws + at[j]) = v[j];
  }
  __syncthreads();

  if (16 * sblk >= p.M) return;
  switch ((p.N + 15) >> 4) {
    case 1: fwd_skinny_tile<1>(p, sblk, piece, ws, pk); break;
    case 2: fwd_skinny_tile<2>(p, sblk, piece, ws, pk); break;
    case 3: fwd_skinny_tile<3>(p, sblk, piece, ws, pk); break;
    case 4: fwd_skinny_tile<4>(p, sblk, piece, ws, pk); break;
    case 5: fwd_skinny_tile<5>(p, sblk, piece, ws, pk); break;
    case 6: fwd_skinny_tile<6>(p, sblk, piece, ws, pk); break;
    case 7: fwd_skinny_tile<7>(p, sblk, piece, ws, pk); break;
    default: fwd_skinny_tile<8>(p, sblk, piece, ws, pk); break;
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
  return (int64_t)16 * ((N + 15) / 16) * fwd_skinny_pitch(sub_len) * 4;
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
  static bool attr_set = false;   // the same for every device of the process
  if (!attr_set) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fwd_skinny_kernel),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             SKINNY_FWD_LDS);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  return launch_k(fwd_skinny_kernel, dim3((unsigned)(groups * p.nsub)), dim3(SKF_NT),
                  (unsigned)lds, s, p, fwd_skinny_pitch(p.sub_len));
}

}  // namespace nf
