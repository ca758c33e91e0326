// Internal declarations shared by the host runtime and the kernel launchers.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nf {

// Every kernel of the library is launched through launch_k.  While the host
// runtime times one launch by the kernel's own start and end (nf_profile with
// repeats = 1) it sets launch_events to a pair of HIP events, which the
// launch binds to that kernel's dispatch; otherwise both are null and the
// launch is a plain one.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents& launch_events();

// Sets the message nf_last_error returns on this thread.
void set_error_message(const char* msg);

template <class T>
struct same_type {
  using type = T;
};

// args convert to the kernel's parameter types (which alone fix P...); each
// is passed by the address of that converted copy
template <typename... P>
inline hipError_t launch_k(void (*kernel)(P...), dim3 grid, dim3 block, unsigned shmem,
                           hipStream_t s, const typename same_type<P>::type&... args) {
  void* argv[] = {const_cast<void*>(static_cast<const void*>(&args))..., nullptr};
  const LaunchEvents& ev = launch_events();
  return hipExtLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, argv, shmem, s,
                            ev.start, ev.stop, 0);
}

// Epilogue of the tiled MFMA contraction C = A(m,k) * B(k,n).
enum Epilogue : int {
  EPI_FWD_STASH = 0,  // z = C + b[n]; out0 = f(z) (activation), out1 = f'(z)
  EPI_FWD_DELTA = 1,  // z = C + b[n]; out0 = (f(z) - y) * f'(z)  (output delta)
  EPI_FWD_OUT = 2,    // z = C + b[n]; out0 = f(z)              (inference)
  EPI_BWD = 3,        // out0 = C * aux                          (hidden delta)
  EPI_DW_SGD = 4,     // G = C; W -= scale * C; bias sums and update
  EPI_DW_PARTIAL = 5, // partial[split] = C; bias partial sums
  EPI_FWD_PIECE = 6   // forward operands, partial[piece] = C over a piece of the k range
};

// Element types of a network's parameters and per-sample buffers.
enum Dtype : int { DT_F32 = 0, DT_F64 = 1 };

// One launch of the contraction, in element type T (float or double).
// Operand A is read as A(m,k) and operand B as B(k,n); `a_kcontig` /
// `b_kcontig` say whether k is the contiguous index.
template <class T>
struct GemmParamsT {
  const T* A;
  const T* B;
  int64_t lda, ldb;
  int M, N, K;
  // split of the k range into pieces: piece z = shard * nsub + sub covers
  // [shard*shard_len + sub*sub_len, min(that + sub_len, (shard+1)*shard_len))
  int nsub;
  int shard_len, sub_len;
  // epilogue operands
  const T* bias;       // [N]
  const T* aux;        // y (EPI_FWD_DELTA) or f'(z) (EPI_BWD), [M][ldaux]
  int64_t ldaux;
  T* out0;             // [M][ld0]
  int64_t ld0;
  T* out1;             // [M][ld1]
  int64_t ld1;
  T* W;                // EPI_DW_SGD: updated weights [M][ldw] (W = Win - scale * G)
  const T* Win;        // EPI_DW_SGD: weights before the step, same layout
  int64_t ldw;
  T* bvec;             // EPI_DW_SGD: updated biases [M]
  const T* bin;        // EPI_DW_SGD: biases before the step
  T* gbias;            // EPI_DW_SGD: bias tendency [M]
  T* partial;          // EPI_DW_PARTIAL: [nsplit][M][ld0]
  int64_t pstride;
  T* pbias;            // EPI_DW_PARTIAL: [nsplit][M]
  T scale;             // eta / batch
  int act;
};
using GemmParams = GemmParamsT<float>;

// Tile shapes available to the host side.
enum TileShape : int { TILE_128x128 = 0, TILE_64x64 = 1 };

// Row pitches and base addresses that allow 16-byte vector loads must be
// multiples of 16 / sizeof(T) elements and 16-byte aligned.
template <class T>
hipError_t launch_gemm(int epi, int tile, bool a_kcontig, bool b_kcontig, bool a_vec, bool b_vec,
                       int nsplit, const GemmParamsT<T>& p, hipStream_t s);

// Name of the kernel instance launch_gemm picks for these arguments.
const char* gemm_name(int epi, int tile, int dtype);

// Forward contractions split over the k range (EPI_FWD_PIECE) finish here:
// z = sum of the pieces in piece order + b[n], then the forward epilogue
// `epi` (EPI_FWD_STASH, EPI_FWD_DELTA or EPI_FWD_OUT) on z.
template <class T>
struct FwdFoldParamsT {
  const T* partial;                        // [nsplit][M][ldp]
  int64_t pstride, ldp;
  int nsplit, M, N;
  const T* bias;                           // [N]
  int act;
  T* out0;                                 // [M][ld0]
  int64_t ld0;
  T* out1;                                 // EPI_FWD_STASH: f'(z) [M][ld1]
  int64_t ld1;
  const T* aux;                            // EPI_FWD_DELTA: y [M][ldaux]
  int64_t ldaux;
};
template <class T>
hipError_t launch_fwd_fold(int epi, const FwdFoldParamsT<T>& f, hipStream_t s);

// The tendency pieces of up to GEMM_GROUP_MAX layers in one launch
// (EPI_DW_PARTIAL; both operands mn-contiguous, A rows vectorisable, B rows as
// b_vec says), problem q split into nsplit[q] pieces.  The workgroup table is
// filled by the launcher.
constexpr int GEMM_GROUP_MAX = 4;
template <class T>
struct GemmGroupT {
  GemmParamsT<T> p[GEMM_GROUP_MAX];
  int start[GEMM_GROUP_MAX + 1];           // first workgroup of each problem
  int n;                                   // problems
};
template <class T>
hipError_t launch_dw_partial_group(int tile, bool b_vec, const GemmGroupT<T>& g,
                                   const int* nsplit, hipStream_t s);

// The tendency pieces of up to GEMM_GROUP_MAX fp32 layers of at most
// SKINNY_MAX_UNITS units in one launch, operands loaded straight into the
// matrix cores (csrc/nf_skinny.hip); same piece layout as
// launch_dw_partial_group.  Problem q has npieces[q] pieces; start[] is
// filled by the launcher.  Both operands and the piece buffer need 16-byte
// aligned rows with pitches of whole 16-byte vectors.
constexpr int SKINNY_MAX_UNITS = 128;
constexpr int SKINNY_PD = 4;    // k-steps of operand loads in flight
struct SkinnyGroup {
  GemmParamsT<float> p[GEMM_GROUP_MAX];
  int start[GEMM_GROUP_MAX + 1];
  int npieces[GEMM_GROUP_MAX];
  int n;
};
hipError_t launch_dw_skinny_group(SkinnyGroup g, hipStream_t s);
// The same for fp64 layers (input tiles of 32, 16-byte loads of two doubles).
struct SkinnyGroup64 {
  GemmParamsT<double> p[GEMM_GROUP_MAX];
  int start[GEMM_GROUP_MAX + 1];
  int npieces[GEMM_GROUP_MAX];
  int n;
};
hipError_t launch_dw_skinny_group64(SkinnyGroup64 g, hipStream_t s);
// inputs per workgroup tile of the fp32 and fp64 tendency kernels
constexpr int SKINNY_TILE_F32 = 64, SKINNY_TILE_F64 = 32;

// Forward pieces of a fp32 layer of at most SKINNY_MAX_UNITS units (N),
// operands loaded straight into the matrix cores (csrc/nf_skinny.hip):
// partial[piece][m][ld0] = sum over k in piece of A[m][k] B[n][k], pieces
// of sub_len inputs (a multiple of 16 when nsub > 1), nsub of them; A rows
// (lda) and B rows (ldb) 16-byte aligned with K and both pitches multiples
// of 4.  A workgroup holds the piece's slice of B in LDS:
// fwd_skinny_lds_bytes(N, sub_len) must not exceed SKINNY_FWD_LDS.
constexpr int SKINNY_FWD_PD = 8;          // k-groups of sample loads in flight
constexpr int SKINNY_FWD_LDS = 160 * 1024;
int64_t fwd_skinny_lds_bytes(int N, int sub_len);
hipError_t launch_fwd_skinny(const GemmParamsT<float>& p, hipStream_t s);

// Fold the per-piece tendencies of up to FOLD_GROUP_MAX layers in piece order,
// store each sum as the tendency, and write the SGD step W = Win - scale * G,
// b = bin - scale * g (W [M][ldw], b [M]).  Layer q's pieces: nshards shards
// of nsub sub-pieces, weights at partial + piece * pstride, biases at
// pbias + piece * M.  The workgroup table is filled by the launcher.
constexpr int FOLD_GROUP_MAX = 8;
constexpr int FOLD_THREADS = 256;
template <class T>
struct FoldLayerT {
  const T* partial;
  int64_t pstride;
  const T* pbias;
  int nsub, M, N;
  int64_t ldw;
  T* G;
  T* gbias;
  const T* Win;
  const T* bin;
  T* W;
  T* b;
};
template <class T>
struct FoldGroupT {
  FoldLayerT<T> l[FOLD_GROUP_MAX];
  int start[FOLD_GROUP_MAX + 1];           // first workgroup of each layer
  int n;                                   // layers
  int nshards;
  T scale;
};
template <class T>
hipError_t launch_fold_sgd(FoldGroupT<T> g, hipStream_t s);

// ---------------------------------------------------------------------------
// Narrow networks: every layer after the input has at most NARROW_WIDTH units
// (the paper's 784-30-10 MNIST network is one).  A training step is two
// kernels: a per-sample pass (forward, output delta, hidden deltas) and the
// batch tendencies with the SGD step.  Per-sample buffers have pitch
// NARROW_WIDTH and zero padding.
// ---------------------------------------------------------------------------
constexpr int NARROW_MAX_LAYERS = 4;
constexpr int NARROW_WIDTH = 32;
constexpr int NARROW_TILE = 16;       // samples per workgroup of the per-sample pass
// batches up to this size take 4-sample workgroups (enough of them to fill
// the chip); larger ones take NARROW_TILE-sample workgroups
constexpr int NARROW_SMALL_BATCH = 2048;
// the narrow kernels read W_1 and input rows through buffer resources; the
// host keeps those ranges (at most NARROW_WIDTH rows of d_0 values) below
// this many bytes, and offsets at or past it read as zeros
constexpr unsigned NARROW_OOB = 0x40000000u;

// Parameter layout of narrow nets: W_1 is [NARROW_WIDTH][ldw_1] and W_l, l >= 2,
// is [NARROW_WIDTH][NARROW_WIDTH]; biases are NARROW_WIDTH long; rows, columns
// and entries past the layer sizes are zero.  The per-sample kernel reads the
// layers past the last one (up to NARROW_MAX_LAYERS) from a zero block.
//
// fp32 narrow nets also keep W_1 packed twice, in the register layouts the
// matrix-core operands of the per-sample kernels take, so that each wave
// reads its share of W_1 with 16-byte loads of 1 KiB contiguous per
// instruction (the vector memory pipeline spends a fixed time per
// instruction that grows with the rows it touches):
//   W1f (4x4x1 operands): block (t, q) of 64 lanes x float4, t < ceil(d0 / 64),
//       q < 8; lane 4 b + i holds W_1[4 q + i][64 t + 4 b .. 64 t + 4 b + 3];
//   W1i (16x16x4 operands): block (c, h), c < ceil(d0 / 16), h < 2; lane
//       r + 16 g holds W_1[16 h + r][16 c + 4 g .. 16 c + 4 g + 3];
// blocks in index order, entries past d_1 or d_0 zero.  The SGD kernel
// writes both with the updated W_1; after any other change of the
// parameters the host rewrites them (narrow_pack_w1) before the next pass.
constexpr int NARROW_PACK_W1F_BLOCK = 8 * 64 * 4;   // floats per step t (8 blocks)
constexpr int NARROW_PACK_W1I_BLOCK = 2 * 64 * 4;   // floats per chunk c (2 blocks)
inline int64_t narrow_pack_w1f_elems(int d0) { return (int64_t)((d0 + 63) / 64) * NARROW_PACK_W1F_BLOCK; }
inline int64_t narrow_pack_w1i_elems(int d0) { return (int64_t)((d0 + 15) / 16) * NARROW_PACK_W1I_BLOCK; }
template <class T>
struct NarrowFwdParamsT {
  const T* X;                              // [B][d0], d0 % (16 / sizeof(T)) == 0, 16-byte aligned
  const T* Y;                              // [B][d_L] targets (training)
  int B, d0, L;
  int dout;                                // d_L
  int dims[NARROW_MAX_LAYERS + 1];
  int acts[NARROW_MAX_LAYERS];
  const T* W[NARROW_MAX_LAYERS];           // W_l (index l-1), padded as above
  int64_t ldw[NARROW_MAX_LAYERS];
  const T* bias[NARROW_MAX_LAYERS];
  T* A[NARROW_MAX_LAYERS];                 // f(z_l) [B][32], l = 1..L-1
  T* D[NARROW_MAX_LAYERS];                 // delta_l [B][32], l = 1..L
  T* out;                                  // inference: f(z_L) [B][d_L]
  int ncu;                                 // compute units of the device
  const T* W1f;                            // packed W_1 (fp32 only), see above
  const T* W1i;
};
using NarrowFwdParams = NarrowFwdParamsT<float>;

template <class T>
struct NarrowDwParamsT {
  int B, L;                                // batch, layers
  int dims[NARROW_MAX_LAYERS + 1];
  const T* X;                              // layer-1 inputs [B][d0]
  const T* A[NARROW_MAX_LAYERS];           // f(z_l) [B][32], l = 1..L-1
  const T* D[NARROW_MAX_LAYERS];           // delta_l [B][32]
  const T* Win[NARROW_MAX_LAYERS];         // parameters before the step
  const T* bin[NARROW_MAX_LAYERS];
  T* W[NARROW_MAX_LAYERS];                 // parameters after the step
  int64_t ldw[NARROW_MAX_LAYERS];
  T* bias[NARROW_MAX_LAYERS];
  T* G[NARROW_MAX_LAYERS];                 // tendencies, same layout as W / bias
  T* gb[NARROW_MAX_LAYERS];
  int tile_base[NARROW_MAX_LAYERS + 1];    // first (16-column, 16-unit) tile of each layer;
                                           // ntiles for the layers past the last one
  int ntiles;                              // tiles of all layers
  T scale;
  T* W1f;                                  // packed copies of the updated W_1 (fp32 only)
  T* W1i;
};
using NarrowDwParams = NarrowDwParamsT<float>;

// The per-sample kernels: 4-sample tiles (batches up to NARROW_SMALL_BATCH),
// 16-sample tiles, and the persistent inference kernel (larger batches).
enum NarrowKernel : int { NK_FWD4 = 0, NK_FWD16 = 1, NK_INFER = 2 };
NarrowKernel narrow_fwd_kernel(bool train, const NarrowFwdParams& p);
hipError_t launch_narrow_fwd(bool train, const NarrowFwdParams& p, hipStream_t s);
// Name of the kernel launch_narrow_fwd picks for this pass.
const char* narrow_fwd_name(bool train, const NarrowFwdParams& p);
hipError_t launch_narrow_dw(const NarrowDwParams& p, hipStream_t s);
// Writes both packed copies of W_1 ([d1][ldw] fp32, rows and columns past
// d1 and d0 taken as zero) into W1f and W1i.
hipError_t launch_narrow_pack_w1(const float* W1, int64_t ldw, int d1, int d0, float* W1f,
                                 float* W1i, hipStream_t s);

// The fp64 counterparts (16-sample tiles for every batch; no persistent
// inference kernel).  Input rows need an even width.
hipError_t launch_narrow64_fwd(bool train, const NarrowFwdParamsT<double>& p, hipStream_t s);
const char* narrow64_fwd_name(bool train, const NarrowFwdParamsT<double>& p);
hipError_t launch_narrow64_dw(const NarrowDwParamsT<double>& p, hipStream_t s);

// ---------------------------------------------------------------------------
// Medium networks (fp32 and fp64): 2..MEDIUM_MAX_LAYERS layers, every layer after the
// input at most MEDIUM_WIDTH units, the weights of layers 2..L within
// MEDIUM_LDS_WEIGHTS floats of LDS as padded below.  Layer 1's contraction
// writes its k pieces; one per-sample kernel does the rest of the forward
// pass and every delta.
// ---------------------------------------------------------------------------
constexpr int MEDIUM_MAX_LAYERS = 4;
constexpr int MEDIUM_WIDTH = 128;
constexpr int MEDIUM_LDS_WEIGHTS = 24576;
// every per-sample buffer the medium pass reads or writes ([np][B][ldz],
// [B][d_L], [B][lda_l]) spans fewer bytes than this: offsets at or past it
// address nothing, so lanes off the tile load zeros and drop their stores
constexpr unsigned MEDIUM_OOB = 0x7fff0000u;

template <class T>
struct MediumParamsT {
  int B, L;
  int dims[MEDIUM_MAX_LAYERS + 1];
  int acts[MEDIUM_MAX_LAYERS];
  const T* zp;                             // layer 1's pieces [np][B][ldz]
  int64_t zstride, ldz;
  int np;
  const T* W[MEDIUM_MAX_LAYERS];           // W_l (index l-1), device layout
  int64_t ldw[MEDIUM_MAX_LAYERS];
  const T* bias[MEDIUM_MAX_LAYERS];
  const T* Y;                              // targets [B][d_L]
  T* A[MEDIUM_MAX_LAYERS];                 // f(z_l) [B][lda_l], l = 1..L-1
  T* D[MEDIUM_MAX_LAYERS];                 // delta_l [B][lda_l], l = 1..L
  int64_t lda[MEDIUM_MAX_LAYERS];
  // W_l, l >= 2, in LDS at woff[l-1] as wrows[l-1] = round_up(d_l, 16) rows
  // of wp[l-1] elements (round_up(d_{l-1}, 16) plus bank padding, 18 mod 32),
  // zero past the layer sizes
  int woff[MEDIUM_MAX_LAYERS], wrows[MEDIUM_MAX_LAYERS], wp[MEDIUM_MAX_LAYERS];
};
using MediumParams = MediumParamsT<float>;
using MediumParams64 = MediumParamsT<double>;
// fp64 nets: the staged weights in at most this many doubles (the tile is
// then one 16-sample block, so the weights and the tile fit in LDS together)
constexpr int MEDIUM64_LDS_WEIGHTS = 15360;
template <class T>
hipError_t launch_medium(const MediumParamsT<T>& p, int ncu, hipStream_t s);

// Adds to *count the number of rows s < n for which out[s][0..d) and
// y[s][0..d) have their first largest entry at the same index (rows holding a
// NaN never count).  Row pitches ldo and ldy in elements.
template <class T>
hipError_t launch_count_correct(const T* out, int64_t ldo, const T* y, int64_t ldy, int64_t n,
                                int d, unsigned long long* count, hipStream_t s);

}  // namespace nf
