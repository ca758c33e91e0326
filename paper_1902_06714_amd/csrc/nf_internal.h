// Internal declarations shared by the host runtime and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nf {

// Epilogue of the tiled fp32 MFMA contraction C = A(m,k) * B(k,n).
enum Epilogue : int {
  EPI_FWD_STASH = 0,  // z = C + b[n]; out0 = f(z) (activation), out1 = f'(z)
  EPI_FWD_DELTA = 1,  // z = C + b[n]; out0 = (f(z) - y) * f'(z)  (output delta)
  EPI_FWD_OUT = 2,    // z = C + b[n]; out0 = f(z)              (inference)
  EPI_BWD = 3,        // out0 = C * aux                          (hidden delta)
  EPI_DW_SGD = 4,     // G = C; W -= scale * C; bias sums and update
  EPI_DW_PARTIAL = 5  // partial[split] = C; bias partial sums
};

// One launch of the contraction.  Operand A is read as A(m,k) and operand B
// as B(k,n); `a_kcontig` / `b_kcontig` say whether k is the contiguous index.
struct GemmParams {
  const float* A;
  const float* B;
  int64_t lda, ldb;
  int M, N, K;
  // split of the k range into pieces: piece z = shard * nsub + sub covers
  // [shard*shard_len + sub*sub_len, min(that + sub_len, (shard+1)*shard_len))
  int nsub;
  int shard_len, sub_len;
  // epilogue operands
  const float* bias;   // [N]
  const float* aux;    // y (EPI_FWD_DELTA) or f'(z) (EPI_BWD), [M][ldaux]
  int64_t ldaux;
  float* out0;         // [M][ld0]
  int64_t ld0;
  float* out1;         // [M][ld1]
  int64_t ld1;
  float* W;            // EPI_DW_SGD: weights [M][ldw] updated in place
  int64_t ldw;
  float* bvec;         // EPI_DW_SGD: biases [M] updated in place
  float* gbias;        // EPI_DW_SGD: bias tendency [M]
  float* partial;      // EPI_DW_PARTIAL: [nsplit][M][ld0]
  int64_t pstride;
  float* pbias;        // EPI_DW_PARTIAL: [nsplit][M]
  float scale;         // eta / batch
  int act;
};

// Tile shapes available to the host side.
enum TileShape : int { TILE_128x128 = 0, TILE_64x64 = 1 };

hipError_t launch_gemm(int epi, int tile, bool a_kcontig, bool b_kcontig, bool a_vec,
                       bool b_vec, int nsplit, const GemmParams& p, hipStream_t s);

// Name of the kernel instance launch_gemm picks for these arguments.
const char* gemm_name(int epi, int tile);

// Fold the per-piece tendencies of one layer in piece order, store the sum as
// the tendency, and apply the SGD step to W [M][ldw] and b [M].
hipError_t launch_fold_sgd(const float* partial, int64_t pstride, const float* pbias,
                           int nshards, int nsub, int M, int N, int64_t ldw, float* G,
                           float* gbias, float* W, float* b, float scale, hipStream_t s);

}  // namespace nf
