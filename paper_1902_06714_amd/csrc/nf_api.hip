// Host runtime behind include/nf.h: argument validation, the device layout of
// a network, its workspace, and the launch sequence of one training step, in
// the network's element type (fp32 or fp64).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <exception>
#include <mutex>
#include <new>
#include <string>
#include <type_traits>
#include <vector>

#include "nf.h"
#include "nf_internal.h"
#include "nf_split.h"

namespace {
thread_local std::string g_err;
}  // namespace

namespace nf {
LaunchEvents& launch_events() {
  thread_local LaunchEvents ev;
  return ev;
}
void set_error_message(const char* msg) { g_err = msg; }
}  // namespace nf

namespace {

nf_status fail(nf_status st, const std::string& msg) {
  g_err = msg;
  return st;
}

nf_status hip_fail(hipError_t e, const char* what) {
  return fail(NF_EDEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

constexpr int64_t kAlign = 64;  // elements between tensors (256 bytes in fp32)

int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

struct LayerLayout {
  int in = 0, out = 0, act = 0;
  int64_t ldw = 0;    // row pitch of W_l (elements), multiple of 4; padding is zero
  int64_t w_off = 0;  // offsets in elements inside the parameter / tendency buffers
  int64_t b_off = 0;
  int64_t lda = 0;    // row pitch of the per-sample buffers of this layer
};

// Restores the caller's current device on scope exit.
struct DeviceGuard {
  int prev = -1;
  bool ok = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) return;
    ok = (prev == dev) || hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

template <class T>
constexpr int dtype_of() {
  return sizeof(T) == 8 ? nf::DT_F64 : nf::DT_F32;
}

}  // namespace

struct nf_net {
  int device = 0;
  int ncu = 0;                 // compute units of the device
  int dtype = nf::DT_F32;
  size_t esz = sizeof(float);  // bytes per element
  std::vector<int> dims;
  std::vector<LayerLayout> layers;
  int64_t n_params = 0;       // canonical elements
  int64_t dev_elems = 0;      // device layout elements
  // parameters, double-buffered: a step reads pbuf[cur] and writes the
  // updated parameters to pbuf[cur ^ 1], then cur flips
  void* pbuf[2] = {nullptr, nullptr};
  int cur = 0;
  void* grads = nullptr;      // device layout, tendencies of the last step
  // workspace for up to ws_batch samples
  int64_t ws_batch = 0;
  void* ws = nullptr;
  std::vector<void*> actv;    // actv[l]: f(z_l) [B][lda_l], l = 1..L-1
  std::vector<void*> fbuf;    // fbuf[l]: f'(z_l) [B][lda_l], l = 1..L-1
  std::vector<void*> dbuf;    // dbuf[l]: delta_l [B][lda_l], l = 1..L
  // per-piece tendencies
  void* partial = nullptr;
  int64_t partial_elems = 0;
  // accuracy: network outputs of one chunk of samples, and the correct count
  void* evalbuf = nullptr;
  int64_t eval_elems = 0;
  unsigned long long* dcount = nullptr;
  // nets of at most NARROW_MAX_LAYERS layers whose every layer after the input
  // has at most NARROW_WIDTH units
  bool narrow = false;
  // narrow nets: offset of a zero block (NARROW_WIDTH^2 weights, then
  // NARROW_WIDTH biases) that stands in for the layers past the last one
  int64_t zero_off = 0;
  // fp32 narrow nets: W_1 packed in the per-sample kernels' operand layouts
  // (W1f, then W1i; see NarrowFwdParamsT), valid for the parameters of
  // version packver; pver counts every change of the current parameters
  void* w1pack = nullptr;
  int64_t w1f_elems = 0;
  uint64_t pver = 1, packver = 0;
  hipStream_t last = nullptr;
  bool used = false;
  // samples whose f'(z_l), l < L, the last training step left in fbuf (0 when
  // that step kept f' in registers, or the workspace has been replaced since)
  int64_t stash_batch = 0;
  // true while a step runs on the shared scratch (nf_train_batch_noalloc):
  // the workspace pointers then point into it and nothing may be allocated
  bool borrowed = false;
  // per-kernel timing (nf_profile)
  struct Rec {
    const char* name;
    hipEvent_t a, b;
    double bytes, flops;
    int repeats;
  };
  int prof = 0;                // 0: off; R >= 1: each kernel runs R times between its events
  std::vector<Rec> recs;
};

namespace {

int num_layers(const nf_net* n) { return (int)n->dims.size() - 1; }

// parameters read by this step, and the buffer its update is written to
template <class T>
T* cur_params(const nf_net* n) {
  return static_cast<T*>(n->pbuf[n->cur]);
}
template <class T>
T* next_params(const nf_net* n) {
  return static_cast<T*>(n->pbuf[n->cur ^ 1]);
}
template <class T>
T* as(void* p) {
  return static_cast<T*>(p);
}

nf_status sync_net(nf_net* n) {
  if (!n->used) return NF_OK;
  hipError_t e = hipStreamSynchronize(n->last);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  return NF_OK;
}

// the parameter buffers, the tendencies and the packed copies of W_1
void free_params(nf_net* n) {
  for (void*& b : n->pbuf) {
    if (b) (void)hipFree(b);
    b = nullptr;
  }
  if (n->grads) (void)hipFree(n->grads);
  if (n->w1pack) (void)hipFree(n->w1pack);
  n->grads = nullptr;
  n->w1pack = nullptr;
}

void free_ws(nf_net* n) {
  if (n->ws) (void)hipFree(n->ws);
  n->ws = nullptr;
  n->ws_batch = 0;
  n->stash_batch = 0;
  n->actv.assign(n->dims.size(), nullptr);
  n->fbuf.assign(n->dims.size(), nullptr);
  n->dbuf.assign(n->dims.size(), nullptr);
}

// The per-sample workspace of `batch` samples: for l < L, f(z_l) and f'(z_l),
// and delta_l for every l, each [batch][lda_l], at the element offsets
// written to aoff/foff/doff (-1 where a layer has none).  Returns the total.
int64_t ws_layout(const nf_net* n, int64_t batch, std::vector<int64_t>* aoff,
                  std::vector<int64_t>* foff, std::vector<int64_t>* doff) {
  const int L = num_layers(n);
  aoff->assign(L + 1, -1);
  foff->assign(L + 1, -1);
  doff->assign(L + 1, -1);
  int64_t total = 0;
  for (int l = 1; l <= L; ++l) {
    const int64_t sz = round_up(batch * n->layers[l].lda, kAlign);
    if (l < L) {
      (*aoff)[l] = total;
      total += sz;
      (*foff)[l] = total;
      total += sz;
    }
    (*doff)[l] = total;
    total += sz;
  }
  return total;
}

// points the net's per-sample buffers at base (element offsets as above)
void ws_assign(nf_net* n, char* base, const std::vector<int64_t>& aoff,
               const std::vector<int64_t>& foff, const std::vector<int64_t>& doff) {
  const int L = num_layers(n);
  for (int l = 1; l <= L; ++l) {
    n->actv[l] = aoff[l] >= 0 ? base + aoff[l] * n->esz : nullptr;
    n->fbuf[l] = foff[l] >= 0 ? base + foff[l] * n->esz : nullptr;
    n->dbuf[l] = base + doff[l] * n->esz;
  }
}

// Make room for `batch` samples.  Growing waits for the net's earlier work,
// which may still read the old buffers.  A net borrowing the shared scratch
// (nf_train_batch_noalloc) never grows: its room was checked beforehand.
nf_status ensure_ws(nf_net* n, int64_t batch) {
  if (batch <= n->ws_batch) return NF_OK;
  if (n->borrowed) return fail(NF_EINVAL, "internal: the scratch workspace is too small");
  nf_status st = sync_net(n);
  if (st != NF_OK) return st;
  std::vector<int64_t> aoff, foff, doff;
  const int64_t total = ws_layout(n, batch, &aoff, &foff, &doff);
  void* buf = nullptr;
  hipError_t e = hipMalloc(&buf, (size_t)total * n->esz);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(NF_ENOMEM,
                "hipMalloc of the workspace failed: " + std::string(hipGetErrorString(e)));
  }
  e = hipMemset(buf, 0, (size_t)total * n->esz);  // pitch padding must read as zero
  if (e != hipSuccess) {
    (void)hipFree(buf);
    return hip_fail(e, "hipMemset");
  }
  free_ws(n);
  n->ws = buf;
  n->ws_batch = batch;
  ws_assign(n, static_cast<char*>(buf), aoff, foff, doff);
  return NF_OK;
}

nf_status ensure_partial(nf_net* n, int64_t elems) {
  if (elems <= n->partial_elems) return NF_OK;
  if (n->borrowed) return fail(NF_EINVAL, "internal: the scratch piece buffer is too small");
  nf_status st = sync_net(n);
  if (st != NF_OK) return st;
  void* buf = nullptr;
  hipError_t e = hipMalloc(&buf, (size_t)elems * n->esz);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(NF_ENOMEM, "hipMalloc of the piece buffer failed");
  }
  if (n->partial) (void)hipFree(n->partial);
  n->partial = buf;
  n->partial_elems = elems;
  return NF_OK;
}

// rows of pitch ld starting at p can be read with aligned 16-byte loads
template <class T>
bool vec_ok(const T* p, int64_t ld) {
  return ld % (int64_t)(16 / sizeof(T)) == 0 && (reinterpret_cast<uintptr_t>(p) & 15) == 0;
}

int pick_tile(int64_t M, int64_t N, int64_t splits) {
  const int64_t big = ((M + 127) / 128) * ((N + 127) / 128) * splits;
  return big >= 256 ? nf::TILE_128x128 : nf::TILE_64x64;
}

void clear_recs(nf_net* n) {
  for (auto& r : n->recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  n->recs.clear();
}

// Runs `enqueue` (one kernel launch) on stream s.  With recording on, the
// launch is timed by a pair of events: for R = 1 the events are bound to the
// kernel's own dispatch (its start and end timestamps, no marker between
// launches); for R > 1 they are recorded on the stream around R back-to-back
// runs of the launch (every kernel reads only buffers it does not write, so
// a repeat recomputes the same values) and the record is charged the average.
template <class F>
nf_status timed(nf_net* n, const char* name, double bytes, double flops, hipStream_t s,
                F&& enqueue) {
  nf_net::Rec r{name, nullptr, nullptr, bytes, flops, n->prof};
  auto drop = [&] {
    if (r.a) (void)hipEventDestroy(r.a);
    if (r.b) (void)hipEventDestroy(r.b);
  };
  if (n->prof) {
    hipError_t e = hipEventCreate(&r.a);
    if (e == hipSuccess) e = hipEventCreate(&r.b);
    if (e == hipSuccess && n->prof > 1) e = hipEventRecord(r.a, s);
    if (e != hipSuccess) {
      drop();
      return hip_fail(e, "profiling event");
    }
  }
  const int reps = n->prof > 1 ? n->prof : 1;
  nf::LaunchEvents& ev = nf::launch_events();
  for (int i = 0; i < reps; ++i) {
    if (n->prof == 1) ev = {r.a, r.b};
    hipError_t e = enqueue();
    ev = {};
    if (e != hipSuccess) {
      drop();
      return hip_fail(e, "kernel launch");
    }
  }
  if (n->prof > 1) {
    hipError_t e = hipEventRecord(r.b, s);
    if (e != hipSuccess) {
      drop();
      return hip_fail(e, "profiling event");
    }
  }
  if (n->prof) n->recs.push_back(r);
  return NF_OK;
}

// Algorithmic bytes of one contraction launch: each operand read once, each
// result written once (esz bytes per element).
double gemm_bytes(int epi, int M_, int N_, int K_, int nsplit, double esz) {
  const double M = M_, N = N_, K = K_;
  switch (epi) {
    case nf::EPI_FWD_STASH: return esz * (M * K + N * K + N + 2 * M * N);
    case nf::EPI_FWD_DELTA: return esz * (M * K + N * K + N + 2 * M * N);
    case nf::EPI_FWD_OUT: return esz * (M * K + N * K + N + M * N);
    case nf::EPI_BWD: return esz * (M * K + K * N + 2 * M * N);
    case nf::EPI_DW_SGD: return esz * (K * M + K * N + 3 * M * N + 3 * M);
    case nf::EPI_FWD_PIECE: return esz * (M * K + N * K + nsplit * M * N);
    default: return esz * (K * M + K * N + nsplit * (M * N + M));
  }
}

// tile_override: a TileShape, or -1 to pick one from the grid size
template <class T>
nf_status launch(nf_net* n, int epi, bool akc, bool bkc, bool av, bool bv, int nsplit,
                 const nf::GemmParamsT<T>& p, hipStream_t s, int tile_override = -1) {
  const int tile = tile_override >= 0 ? tile_override : pick_tile(p.M, p.N, nsplit);
  return timed(n, nf::gemm_name(epi, tile, dtype_of<T>()),
               gemm_bytes(epi, p.M, p.N, p.K, nsplit, (double)sizeof(T)),
               2.0 * p.M * (double)p.N * p.K, s,
               [&] { return nf::launch_gemm<T>(epi, tile, akc, bkc, av, bv, nsplit, p, s); });
}

// The cut of a forward contraction (M samples, N units, K inputs) over its
// k range: one piece unless the 64 x 64 tile grid is under twice the CU count
// and K >= 256 (general nets take it only when the grid would use the
// 64 x 64 tile anyway).  Pieces start on whole 16-input stages, so a vector
// load never reaches into the next piece and every piece start stays 16-byte
// aligned (nf_split.h).
nf::KSplit fwd_split(const nf_net* n, int64_t M, int64_t N, int64_t K, bool small_tile_only) {
  const int64_t tiles = ((M + 63) / 64) * ((N + 63) / 64);
  const int64_t want = 2 * (int64_t)(n->ncu > 0 ? n->ncu : 256);
  if ((small_tile_only && pick_tile(M, N, 1) != nf::TILE_64x64) || tiles >= want || K < 256)
    return nf::KSplit{1, (int)K};
  const int64_t nsplit = std::min<int64_t>({(want + tiles - 1) / tiles, K / 128, 16});
  return nf::k_split(K, nsplit);
}

// The k pieces of the skinny forward kernel (layers of at most
// SKINNY_MAX_UNITS units): one workgroup per (128 samples, piece) holding the
// piece's slice of W in LDS, one workgroup per CU.  Among the piece counts
// whose slice fits in LDS, the one with the fewest k-groups on the busiest
// CU wins, the smaller on ties; nsplit 0 when none fits.
nf::KSplit fwd_skinny_split(const nf_net* n, int64_t M, int64_t N, int64_t K) {
  const int64_t ncu = n->ncu > 0 ? n->ncu : 256;
  const int64_t groups = (M + 127) / 128;
  nf::KSplit best{0, 0};
  int64_t best_cost = -1;
  for (int want = 1; want <= 16; ++want) {
    const nf::KSplit ks = nf::k_split(K, want);
    if (nf::fwd_skinny_lds_bytes((int)N, ks.sub_len) > nf::SKINNY_FWD_LDS) continue;
    const int64_t per_cu = (groups * ks.nsplit + ncu - 1) / ncu;
    const int64_t cost = per_cu * ((ks.sub_len + 15) / 16);
    if (best_cost < 0 || cost < best_cost) {
      best = ks;
      best_cost = cost;
    }
  }
  return best;
}

// layer 1 of the medium path goes to the skinny forward kernel
template <class T>
bool medium_fwd_skinny(const nf_net* n, const T* x, int64_t batch) {
  if constexpr (sizeof(T) != 4) {
    return false;
  } else {
    const LayerLayout& l1 = n->layers[1];
    return l1.out <= nf::SKINNY_MAX_UNITS && vec_ok(x, n->dims[0]) &&
           fwd_skinny_split(n, batch, l1.out, l1.in).nsplit > 0;
  }
}

// elements of the pieces of a forward contraction cut into nsplit pieces
int64_t fwd_piece_elems(int64_t M, int64_t N, int nsplit) {
  return nsplit <= 1 ? 0 : nsplit * round_up(M * round_up(N, 4), kAlign);
}

// The tendency pieces of a step: each layer whose batch is split (shards, or
// sub-pieces when the tile grid alone would leave most compute units idle)
// gets a region of the piece buffer, the weights' pieces [pieces][d_l][ldw_l]
// followed by the biases' pieces.  Returns the elements of all the regions.
struct DwPiece {
  int l, nsub;
  int64_t pstride, off;                  // weights' pitch per piece, region offset
};

// Layers that the skinny tendency kernels take (at most SKINNY_MAX_UNITS
// units) share one launch of equal workgroups, one per (piece, input tile of
// 64 in fp32, 32 in fp64); they get one common sub-piece count, doubled only
// while the doubled launch still fits two workgroups per CU (the kernel's
// occupancy), so that no CU runs a workgroup after the others are done.
// Other layers' pieces are sized by the 128 x 128 tiles of the general
// kernel.
bool dw_skinny_layer(const nf_net* n, int l) {
  return n->layers[l].out <= nf::SKINNY_MAX_UNITS;
}

int64_t dw_plan(const nf_net* n, int64_t batch, int shards, std::vector<DwPiece>* pieces) {
  const int L = num_layers(n);
  const int64_t shard_len = batch / shards;
  const int64_t ncu = n->ncu > 0 ? n->ncu : 256;
  int64_t skinny_wg = 0;
  const int64_t tile = n->dtype == nf::DT_F32 ? nf::SKINNY_TILE_F32 : nf::SKINNY_TILE_F64;
  for (int l = 1; l <= L; ++l)
    if (dw_skinny_layer(n, l)) skinny_wg += (n->layers[l].in + tile - 1) / tile * shards;
  int skinny_nsub = 1;
  while (skinny_wg * skinny_nsub * 2 <= 2 * ncu && shard_len / (skinny_nsub * 2) >= 256 &&
         skinny_nsub < 64 && (int64_t)shards * skinny_nsub * 2 <= 65535)
    skinny_nsub *= 2;
  int64_t total = 0;
  pieces->clear();
  for (int l = L; l >= 1; --l) {
    const LayerLayout& ly = n->layers[l];
    const int64_t M = ly.out, N = ly.in;
    int nsub = 1;
    const int64_t tiles = ((M + 127) / 128) * ((N + 127) / 128);
    if (dw_skinny_layer(n, l))
      nsub = skinny_nsub;
    else
      while (tiles * shards * nsub < 256 && shard_len / (nsub * 2) >= 256 && nsub < 64 &&
             (int64_t)shards * nsub * 2 <= 65535)
        nsub *= 2;
    if (shards * nsub == 1) continue;
    const int64_t pstride = round_up(M * ly.ldw, kAlign);
    const int64_t nsplit = (int64_t)shards * nsub;
    pieces->push_back({l, nsub, pstride, total});
    total += round_up(nsplit * (pstride + round_up(M, kAlign)), kAlign);
  }
  return total;
}

// Forward propagation of `batch` samples through every layer (section 3.2).
// train: keep f(z_l) and f'(z_l) for back-propagation and finish with the
// output delta; otherwise write f(z_L) to `out`.
template <class T>
nf_status run_forward(nf_net* n, const T* x, const T* y, int64_t batch, T* out, bool train,
                      hipStream_t s) {
  const int L = num_layers(n);
  for (int l = 1; l <= L; ++l) {
    const LayerLayout& ly = n->layers[l];
    nf::GemmParamsT<T> p{};
    p.A = l == 1 ? x : as<T>(n->actv[l - 1]);
    p.lda = l == 1 ? n->dims[0] : n->layers[l - 1].lda;
    p.B = cur_params<T>(n) + ly.w_off;
    p.ldb = ly.ldw;
    p.M = (int)batch;
    p.N = ly.out;
    p.K = ly.in;
    p.nsub = 1;
    p.bias = cur_params<T>(n) + ly.b_off;
    p.act = ly.act;
    const bool av = l == 1 ? vec_ok(x, n->dims[0]) : true;
    int epi;
    if (train) {
      if (l < L) {
        epi = nf::EPI_FWD_STASH;
        p.out0 = as<T>(n->actv[l]);
        p.ld0 = ly.lda;
        p.out1 = as<T>(n->fbuf[l]);
        p.ld1 = ly.lda;
      } else {
        epi = nf::EPI_FWD_DELTA;
        p.aux = y;
        p.ldaux = ly.out;
        p.out0 = as<T>(n->dbuf[l]);
        p.ld0 = ly.lda;
      }
    } else {
      epi = nf::EPI_FWD_OUT;
      if (l < L) {
        p.out0 = as<T>(n->actv[l]);
        p.ld0 = ly.lda;
      } else {
        p.out0 = out;
        p.ld0 = ly.out;
      }
    }
    // A contraction with too few 64 x 64 tiles to fill the chip and a long k
    // range is split over the k range; a fold adds the pieces in order and
    // applies the epilogue.
    const nf::KSplit ks = fwd_split(n, p.M, p.N, p.K, true);
    int nsplit = ks.nsplit;
    nf_status st;
    if (nsplit <= 1) {
      st = launch<T>(n, epi, true, true, av, true, 1, p, s);
    } else {
      const int sub_len = ks.sub_len;
      const int64_t ldp = round_up(p.N, 4);
      const int64_t pstride = round_up((int64_t)p.M * ldp, kAlign);
      st = ensure_partial(n, nsplit * pstride);
      if (st != NF_OK) return st;
      nf::GemmParamsT<T> q = p;
      q.shard_len = p.K;
      q.nsub = nsplit;
      q.sub_len = sub_len;
      q.partial = as<T>(n->partial);
      q.pstride = pstride;
      q.ld0 = ldp;
      st = launch<T>(n, nf::EPI_FWD_PIECE, true, true, av, true, nsplit, q, s, nf::TILE_64x64);
      if (st != NF_OK) return st;
      nf::FwdFoldParamsT<T> f{};
      f.partial = q.partial;
      f.pstride = pstride;
      f.ldp = ldp;
      f.nsplit = nsplit;
      f.M = p.M;
      f.N = p.N;
      f.bias = p.bias;
      f.act = p.act;
      f.out0 = p.out0;
      f.ld0 = p.ld0;
      f.out1 = p.out1;
      f.ld1 = p.ld1;
      f.aux = p.aux;
      f.ldaux = p.ldaux;
      const double mn = (double)p.M * p.N;
      const double outs = epi == nf::EPI_FWD_STASH ? 2.0 : (epi == nf::EPI_FWD_DELTA ? 2.0 : 1.0);
      st = timed(n, sizeof(T) == 8 ? "fwd64_fold" : "fwd_fold",
                 (double)sizeof(T) * (mn * (nsplit + outs) + p.N), mn * (nsplit + 1), s,
                 [&] { return nf::launch_fwd_fold<T>(epi, f, s); });
    }
    if (st != NF_OK) return st;
  }
  return NF_OK;
}

// Back-propagation and the SGD step (sections 3.3-3.5).  Layer l's weights are
// updated only after delta_{l-1}, which reads them, has been formed.
template <class T>
nf_status run_backward_update(nf_net* n, const T* x, int64_t batch, double eta, int shards,
                              hipStream_t s, bool deltas_done = false) {
  const int L = num_layers(n);
  const T scale = (T)(eta / (double)batch);
  const int64_t shard_len = batch / shards;
  T* P = cur_params<T>(n);
  T* Q = next_params<T>(n);
  T* G = as<T>(n->grads);

  // Tendencies of layer l: G = delta_l^T A_{l-1}, g = sum of delta_l rows.
  // A batch in one piece takes the kernel with the SGD step fused in; split
  // batches (shards, or sub-pieces when the tile grid alone would leave most
  // compute units idle) write per-piece sums, which are folded in piece order
  // after every layer's pieces are in.  Each layer's pieces get their own
  // region of the workspace, so the piece kernels of several layers share a
  // launch and one fold serves them all.
  using Piece = DwPiece;
  std::vector<Piece> pieces;
  const int64_t total = dw_plan(n, batch, shards, &pieces);
  if (total > 0) {
    nf_status st = ensure_partial(n, total);
    if (st != NF_OK) return st;
  }
  auto piece_of = [&](int l) -> const Piece* {
    for (const Piece& pc : pieces)
      if (pc.l == l) return &pc;
    return nullptr;
  };
  auto dw_params = [&](int l) {
    const LayerLayout& ly = n->layers[l];
    nf::GemmParamsT<T> p{};
    p.A = as<T>(n->dbuf[l]);
    p.lda = ly.lda;
    p.B = l == 1 ? x : as<T>(n->actv[l - 1]);
    p.ldb = l == 1 ? n->dims[0] : n->layers[l - 1].lda;
    p.M = ly.out;
    p.N = ly.in;
    p.K = (int)batch;
    p.shard_len = (int)shard_len;
    p.scale = scale;
    return p;
  };

  for (int l = L; l >= 1; --l) {
    const LayerLayout& ly = n->layers[l];
    if (l > 1 && !deltas_done) {
      // delta_{l-1} = (delta_l W_l) * f'(z_{l-1}), with this step's W_l
      const LayerLayout& lp = n->layers[l - 1];
      nf::GemmParamsT<T> p{};
      p.A = as<T>(n->dbuf[l]);
      p.lda = ly.lda;
      p.B = P + ly.w_off;
      p.ldb = ly.ldw;
      p.M = (int)batch;
      p.N = lp.out;
      p.K = ly.out;
      p.nsub = 1;
      p.aux = as<T>(n->fbuf[l - 1]);
      p.ldaux = lp.lda;
      p.out0 = as<T>(n->dbuf[l - 1]);
      p.ld0 = lp.lda;
      nf_status st = launch<T>(n, nf::EPI_BWD, true, false, true, true, 1, p, s);
      if (st != NF_OK) return st;
    }
    if (!piece_of(l)) {
      const bool bv = l == 1 ? vec_ok(x, n->dims[0]) : true;
      nf::GemmParamsT<T> p = dw_params(l);
      p.nsub = 1;
      p.sub_len = (int)shard_len;
      p.out0 = G + ly.w_off;
      p.ld0 = ly.ldw;
      p.W = Q + ly.w_off;
      p.Win = P + ly.w_off;
      p.ldw = ly.ldw;
      p.bvec = Q + ly.b_off;
      p.bin = P + ly.b_off;
      p.gbias = G + ly.b_off;
      nf_status st = launch<T>(n, nf::EPI_DW_SGD, false, false, true, bv, 1, p, s);
      if (st != NF_OK) return st;
    }
  }
  if (pieces.empty()) return NF_OK;

  // the piece kernels, grouped by tile shape and B-row vector loads (layer
  // order within a group), up to GEMM_GROUP_MAX layers per launch; layers of
  // at most SKINNY_MAX_UNITS units with 16-byte operand rows take the skinny
  // tendency kernel of their element type
  const int dtype = dtype_of<T>();
  std::vector<bool> done(pieces.size(), false);
  auto piece_params = [&](const Piece& pc) {
    const LayerLayout& lj = n->layers[pc.l];
    nf::GemmParamsT<T> p = dw_params(pc.l);
    p.nsub = pc.nsub;
    p.sub_len = (int)((shard_len + pc.nsub - 1) / pc.nsub);
    p.partial = as<T>(n->partial) + pc.off;
    p.pstride = pc.pstride;
    p.ld0 = lj.ldw;
    p.pbias = p.partial + (int64_t)shards * pc.nsub * pc.pstride;
    return p;
  };
  {
    {
      std::conditional_t<sizeof(T) == 4, nf::SkinnyGroup, nf::SkinnyGroup64> g{};
      double bytes = 0.0, flops = 0.0;
      for (size_t j = 0; j < pieces.size() && g.n < nf::GEMM_GROUP_MAX; ++j) {
        const Piece& pj = pieces[j];
        const nf::GemmParamsT<T> p = piece_params(pj);
        if (p.M > nf::SKINNY_MAX_UNITS || !vec_ok(p.A, p.lda) || !vec_ok(p.B, p.ldb)) continue;
        const int nsplit = shards * pj.nsub;
        g.npieces[g.n] = nsplit;
        g.p[g.n++] = p;
        bytes += gemm_bytes(nf::EPI_DW_PARTIAL, p.M, p.N, p.K, nsplit, (double)sizeof(T));
        flops += 2.0 * p.M * (double)p.N * p.K;
        done[j] = true;
      }
      if (g.n > 0) {
        nf_status st;
        if constexpr (sizeof(T) == 4)
          st = timed(n, "dw_skinny", bytes, flops, s,
                     [&] { return nf::launch_dw_skinny_group(g, s); });
        else
          st = timed(n, "dw64_skinny", bytes, flops, s,
                     [&] { return nf::launch_dw_skinny_group64(g, s); });
        if (st != NF_OK) return st;
      }
    }
  }
  for (size_t i = 0; i < pieces.size(); ++i) {
    if (done[i]) continue;
    const Piece& pi = pieces[i];
    const LayerLayout& li = n->layers[pi.l];
    const int tile = pick_tile(li.out, li.in, (int64_t)shards * pi.nsub);
    const bool bv = pi.l == 1 ? vec_ok(x, n->dims[0]) : true;
    nf::GemmGroupT<T> g{};
    int nsplit[nf::GEMM_GROUP_MAX];
    double bytes = 0.0, flops = 0.0;
    for (size_t j = i; j < pieces.size() && g.n < nf::GEMM_GROUP_MAX; ++j) {
      if (done[j]) continue;
      const Piece& pj = pieces[j];
      const LayerLayout& lj = n->layers[pj.l];
      const int tj = pick_tile(lj.out, lj.in, (int64_t)shards * pj.nsub);
      const bool bvj = pj.l == 1 ? vec_ok(x, n->dims[0]) : true;
      if (tj != tile || bvj != bv) continue;
      nf::GemmParamsT<T> p = piece_params(pj);
      nsplit[g.n] = shards * pj.nsub;
      g.p[g.n++] = p;
      bytes += gemm_bytes(nf::EPI_DW_PARTIAL, p.M, p.N, p.K, nsplit[g.n - 1], (double)sizeof(T));
      flops += 2.0 * p.M * (double)p.N * p.K;
      done[j] = true;
    }
    nf_status st = timed(n, nf::gemm_name(nf::EPI_DW_PARTIAL, tile, dtype), bytes, flops, s, [&] {
      return nf::launch_dw_partial_group<T>(tile, bv, g, nsplit, s);
    });
    if (st != NF_OK) return st;
  }

  // one fold for up to FOLD_GROUP_MAX layers
  for (size_t i = 0; i < pieces.size(); i += nf::FOLD_GROUP_MAX) {
    nf::FoldGroupT<T> f{};
    f.nshards = shards;
    f.scale = scale;
    double bytes = 0.0, flops = 0.0;
    for (size_t j = i; j < pieces.size() && f.n < nf::FOLD_GROUP_MAX; ++j) {
      const Piece& pc = pieces[j];
      const LayerLayout& ly = n->layers[pc.l];
      const int64_t nsplit = (int64_t)shards * pc.nsub;
      nf::FoldLayerT<T>& fl = f.l[f.n++];
      fl.partial = as<T>(n->partial) + pc.off;
      fl.pstride = pc.pstride;
      fl.pbias = fl.partial + nsplit * pc.pstride;
      fl.nsub = pc.nsub;
      fl.M = ly.out;
      fl.N = ly.in;
      fl.ldw = ly.ldw;
      fl.G = G + ly.w_off;
      fl.gbias = G + ly.b_off;
      fl.Win = P + ly.w_off;
      fl.bin = P + ly.b_off;
      fl.W = Q + ly.w_off;
      fl.b = Q + ly.b_off;
      const double elems = (double)ly.out * ly.in + ly.out;
      bytes += (double)sizeof(T) * elems * (nsplit + 3);
      flops += elems * (nsplit + 1);
    }
    nf_status st = timed(n, sizeof(T) == 8 ? "fold64_sgd" : "fold_sgd", bytes, flops, s,
                         [&] { return nf::launch_fold_sgd<T>(f, s); });
    if (st != NF_OK) return st;
  }
  return NF_OK;
}

// ---------------------------------------------------------------------------
// narrow networks: the two-kernel step of csrc/nf_narrow.hip (fp32) and
// csrc/nf_narrow64.hip (fp64)
// ---------------------------------------------------------------------------
// input rows must allow 16-byte loads: a width that is a multiple of
// 16 / sizeof(T) elements and a 16-byte aligned base
template <class T>
bool narrow_rows_ok(const nf_net* n, const T* x) {
  return n->narrow && n->dims[0] % (16 / (int)sizeof(T)) == 0 && vec_ok(x, n->dims[0]) &&
         (int64_t)n->dims[0] * nf::NARROW_WIDTH * (int64_t)sizeof(T) < (int64_t)nf::NARROW_OOB;
}

template <class T>
nf::NarrowFwdParamsT<T> narrow_fwd_params(const nf_net* n, const T* x, const T* y, int64_t batch,
                                          T* out) {
  nf::NarrowFwdParamsT<T> p{};
  const int L = num_layers(n);
  T* P = cur_params<T>(n);
  p.X = x;
  p.Y = y;
  p.B = (int)batch;
  p.d0 = n->dims[0];
  p.L = L;
  p.dims[0] = n->dims[0];
  for (int l = 1; l <= nf::NARROW_MAX_LAYERS; ++l) {
    if (l <= L) {
      const LayerLayout& ly = n->layers[l];
      p.dims[l] = ly.out;
      p.acts[l - 1] = ly.act;
      p.W[l - 1] = P + ly.w_off;
      p.ldw[l - 1] = ly.ldw;
      p.bias[l - 1] = P + ly.b_off;
      p.A[l - 1] = as<T>(n->actv[l]);
      p.D[l - 1] = as<T>(n->dbuf[l]);
    } else {
      // zero weights and biases for the layers past the last one
      p.W[l - 1] = P + n->zero_off;
      p.ldw[l - 1] = nf::NARROW_WIDTH;
      p.bias[l - 1] = P + n->zero_off + nf::NARROW_WIDTH * nf::NARROW_WIDTH;
    }
  }
  p.dout = n->dims[L];
  p.out = out;
  p.ncu = n->ncu;
  if constexpr (sizeof(T) == 4) {
    p.W1f = as<T>(n->w1pack);
    p.W1i = as<T>(n->w1pack) + n->w1f_elems;
  }
  return p;
}

// The packed copies of W_1 for the current parameters (fp32 narrow nets):
// rewritten from W_1 unless the last step's SGD kernel wrote them
nf_status ensure_packed(nf_net* n, hipStream_t s) {
  if (!n->w1pack || n->packver == n->pver) return NF_OK;
  const LayerLayout& l1 = n->layers[1];
  float* P = cur_params<float>(n);
  float* W1f = as<float>(n->w1pack);
  nf_status st = timed(n, "narrow_pack_w1", 8.0 * (double)(n->w1f_elems + nf::narrow_pack_w1i_elems(l1.in)),
                       0.0, s, [&] {
                         return nf::launch_narrow_pack_w1(P + l1.w_off, l1.ldw, l1.out, l1.in, W1f,
                                                          W1f + n->w1f_elems, s);
                       });
  if (st == NF_OK) n->packver = n->pver;
  return st;
}

// Algorithmic work of the per-sample pass: inputs, targets and weights read,
// per-sample activations and deltas written; forward and delta flops.
void narrow_fwd_work(const nf_net* n, int64_t B, bool train, double* bytes, double* flops) {
  const int L = num_layers(n);
  double by = (double)B * n->dims[0], fl = 0.0;
  for (int l = 1; l <= L; ++l) {
    const double dl = n->dims[l], dp = n->dims[l - 1];
    by += dl * dp + dl;
    fl += 2.0 * B * dl * dp;
    if (train && l >= 2) fl += 2.0 * B * dl * dp;
  }
  if (train) {
    by += (double)B * n->dims[L];                       // targets
    for (int l = 1; l <= L; ++l) by += (double)B * n->dims[l] * (l < L ? 2 : 1);
  } else {
    by += (double)B * n->dims[L];                       // outputs
  }
  *bytes = (double)n->esz * by;
  *flops = fl;
}

template <class T>
nf_status narrow_train_step(nf_net* n, const T* x, const T* y, int64_t batch, double eta,
                            hipStream_t s) {
  const int L = num_layers(n);
  double by, fl;
  narrow_fwd_work(n, batch, true, &by, &fl);
  const nf::NarrowFwdParamsT<T> fp = narrow_fwd_params<T>(n, x, y, batch, nullptr);
  nf_status st;
  if constexpr (sizeof(T) == 4) {
    st = ensure_packed(n, s);
    if (st != NF_OK) return st;
    st = timed(n, nf::narrow_fwd_name(true, fp), by, fl, s,
               [&] { return nf::launch_narrow_fwd(true, fp, s); });
  }
  else
    st = timed(n, nf::narrow64_fwd_name(true, fp), by, fl, s,
               [&] { return nf::launch_narrow64_fwd(true, fp, s); });
  if (st != NF_OK) return st;

  T* P = cur_params<T>(n);
  T* Q = next_params<T>(n);
  T* G = as<T>(n->grads);
  nf::NarrowDwParamsT<T> dp{};
  dp.B = (int)batch;
  dp.L = L;
  dp.X = x;
  dp.scale = (T)(eta / (double)batch);
  dp.dims[0] = n->dims[0];
  int base = 0;
  double dby = 0.0, dfl = 0.0;
  for (int l = 1; l <= L; ++l) {
    const LayerLayout& ly = n->layers[l];
    dp.dims[l] = ly.out;
    dp.A[l - 1] = l < L ? as<T>(n->actv[l]) : nullptr;
    dp.D[l - 1] = as<T>(n->dbuf[l]);
    dp.Win[l - 1] = P + ly.w_off;
    dp.bin[l - 1] = P + ly.b_off;
    dp.W[l - 1] = Q + ly.w_off;
    dp.ldw[l - 1] = ly.ldw;
    dp.bias[l - 1] = Q + ly.b_off;
    dp.G[l - 1] = G + ly.w_off;
    dp.gb[l - 1] = G + ly.b_off;
    dp.tile_base[l - 1] = base;
    base += (ly.in + 15) / 16 * ((ly.out + 15) / 16);
    // deltas and previous activations read, tendencies written, parameters updated
    const double M = ly.out, N = ly.in;
    dby += (double)sizeof(T) * ((double)batch * (M + N) + 3 * M * N + 3 * M);
    dfl += 2.0 * batch * M * N;
  }
  for (int l = L; l <= nf::NARROW_MAX_LAYERS; ++l) dp.tile_base[l] = base;
  dp.ntiles = base;
  if constexpr (sizeof(T) == 4) {
    dp.W1f = as<T>(n->w1pack);
    dp.W1i = as<T>(n->w1pack) + n->w1f_elems;
  }
  if constexpr (sizeof(T) == 4)
    return timed(n, "narrow_dw_sgd", dby, dfl, s, [&] { return nf::launch_narrow_dw(dp, s); });
  else
    return timed(n, "narrow64_dw_sgd", dby, dfl, s,
                 [&] { return nf::launch_narrow64_dw(dp, s); });
}

// ---------------------------------------------------------------------------
// medium fp32 networks: layer 1's contraction in k pieces, then the
// per-sample kernel of csrc/nf_medium.hip for the rest of the forward pass and
// every delta
// ---------------------------------------------------------------------------
// LDS placement of W_l, l >= 2 (see MediumParams); false when the net or the
// batch does not qualify: every per-sample buffer of the pass (at most 16
// pieces of [batch][<= 128] values) must span fewer than MEDIUM_OOB bytes
template <class T>
bool medium_layout(const nf_net* n, int64_t batch, nf::MediumParamsT<T>* p) {
  const int L = num_layers(n);
  if (n->dtype != dtype_of<T>() || L < 2 || L > nf::MEDIUM_MAX_LAYERS) return false;
  if (batch * 16 * (nf::MEDIUM_WIDTH + 4) * (int64_t)sizeof(T) >= (int64_t)nf::MEDIUM_OOB)
    return false;
  for (int l = 1; l <= L; ++l)
    if (n->dims[l] > nf::MEDIUM_WIDTH) return false;
  int off = 0;
  for (int l = 2; l <= L; ++l) {
    // pitch 18 mod 32 elements: both the row-wise (forward) and the
    // column-wise (delta) operand reads of a half-wave hit distinct banks
    const int cw = (int)round_up(n->dims[l - 1], 16);
    const int rows = (int)round_up(n->dims[l], 16), wp = cw + (cw % 32 == 0 ? 18 : 2);
    p->woff[l - 1] = off;
    p->wrows[l - 1] = rows;
    p->wp[l - 1] = wp;
    off += rows * wp;
  }
  return off <= (sizeof(T) == 4 ? nf::MEDIUM_LDS_WEIGHTS : nf::MEDIUM64_LDS_WEIGHTS);
}

template <class T>
nf_status medium_forward_deltas(nf_net* n, const T* x, const T* y, int64_t batch,
                                hipStream_t s) {
  nf::MediumParamsT<T> mp{};
  if (!medium_layout<T>(n, batch, &mp)) return fail(NF_EINVAL, "internal: not a medium net");
  const int L = num_layers(n);
  const LayerLayout& l1 = n->layers[1];
  T* P = cur_params<T>(n);

  // layer 1: z_1 in k pieces (one piece when the tile grid fills the chip)
  nf::GemmParamsT<T> p{};
  p.A = x;
  p.lda = n->dims[0];
  p.B = P + l1.w_off;
  p.ldb = l1.ldw;
  p.M = (int)batch;
  p.N = l1.out;
  p.K = l1.in;
  const bool skinny = medium_fwd_skinny<T>(n, x, batch);
  const nf::KSplit ks = skinny ? fwd_skinny_split(n, p.M, p.N, p.K) : fwd_split(n, p.M, p.N, p.K, false);
  const int sub_len = ks.sub_len;
  const int nsplit = ks.nsplit;
  const int64_t ldz = round_up(p.N, 4);
  const int64_t zstride = round_up((int64_t)p.M * ldz, kAlign);
  nf_status st = ensure_partial(n, nsplit * zstride);
  if (st != NF_OK) return st;
  p.shard_len = p.K;
  p.nsub = nsplit;
  p.sub_len = sub_len;
  p.partial = as<T>(n->partial);
  p.pstride = zstride;
  p.ld0 = ldz;
  if constexpr (sizeof(T) == 4) {
    if (skinny) {
      st = timed(n, "fwd_skinny", gemm_bytes(nf::EPI_FWD_PIECE, p.M, p.N, p.K, nsplit, 4.0),
                 2.0 * p.M * (double)p.N * p.K, s, [&] { return nf::launch_fwd_skinny(p, s); });
      if (st != NF_OK) return st;
    }
  }
  if (!skinny) {
    const bool av = vec_ok(x, n->dims[0]);
    st = launch<T>(n, nf::EPI_FWD_PIECE, true, true, av, true, nsplit, p, s, nf::TILE_64x64);
    if (st != NF_OK) return st;
  }

  mp.B = (int)batch;
  mp.L = L;
  for (int l = 0; l <= L; ++l) mp.dims[l] = n->dims[l];
  mp.zp = p.partial;
  mp.zstride = zstride;
  mp.ldz = ldz;
  mp.np = nsplit;
  mp.Y = y;
  const double es = (double)sizeof(T);
  double by = es * ((double)nsplit * batch * p.N + (double)batch * n->dims[L]), fl = 0.0;
  for (int l = 1; l <= L; ++l) {
    const LayerLayout& ly = n->layers[l];
    mp.acts[l - 1] = ly.act;
    mp.W[l - 1] = P + ly.w_off;
    mp.ldw[l - 1] = ly.ldw;
    mp.bias[l - 1] = P + ly.b_off;
    mp.A[l - 1] = as<T>(n->actv[l]);
    mp.D[l - 1] = as<T>(n->dbuf[l]);
    mp.lda[l - 1] = ly.lda;
    by += es * ((double)batch * ly.out * (l < L ? 2 : 1) + (l >= 2 ? (double)ly.out * ly.in : 0));
    if (l >= 2) fl += 4.0 * batch * (double)ly.out * ly.in;   // forward and delta products
  }
  return timed(n, sizeof(T) == 4 ? "medium_fwd_deltas" : "medium64_fwd_deltas", by, fl, s,
               [&] { return nf::launch_medium(mp, n->ncu > 0 ? n->ncu : 256, s); });
}

// ---------------------------------------------------------------------------
// the step and inference in element type T
// ---------------------------------------------------------------------------
template <class T>
nf_status train_step(nf_net* n, const T* x, const T* y, int64_t batch, double eta, int shards,
                     hipStream_t s) {
  nf_status st;
  const bool narrow = shards == 1 && narrow_rows_ok<T>(n, x);
  nf::MediumParamsT<T> mp{};
  if (narrow) {
    st = narrow_train_step<T>(n, x, y, batch, eta, s);
  } else if (medium_layout<T>(n, batch, &mp)) {
    st = medium_forward_deltas<T>(n, x, y, batch, s);
    if (st == NF_OK) st = run_backward_update<T>(n, x, batch, eta, shards, s, true);
  } else {
    st = run_forward<T>(n, x, y, batch, nullptr, true, s);
    if (st == NF_OK) st = run_backward_update<T>(n, x, batch, eta, shards, s);
  }
  n->stash_batch = (!narrow && !medium_layout<T>(n, batch, &mp) && st == NF_OK) ? batch : 0;
  // the updated parameters are in the other buffer from here on (a failed
  // launch leaves the net in an undefined state, reported as NF_EDEVICE);
  // the narrow step's SGD kernel has packed its W_1 as well
  if (st == NF_OK) {
    n->cur ^= 1;
    ++n->pver;
    if (narrow) n->packver = n->pver;
  }
  return st;
}

// f(z_L) of `batch` samples into out [batch][d_L] (inference, no stash)
template <class T>
nf_status infer(nf_net* n, const T* x, int64_t batch, T* out, hipStream_t s) {
  nf_status st = ensure_ws(n, batch);
  if (st != NF_OK) return st;
  if (narrow_rows_ok<T>(n, x)) {
    double by, fl;
    narrow_fwd_work(n, batch, false, &by, &fl);
    const nf::NarrowFwdParamsT<T> fp = narrow_fwd_params<T>(n, x, nullptr, batch, out);
    if constexpr (sizeof(T) == 4) {
      st = ensure_packed(n, s);
      if (st != NF_OK) return st;
      return timed(n, nf::narrow_fwd_name(false, fp), by, fl, s,
                   [&] { return nf::launch_narrow_fwd(false, fp, s); });
    }
    else
      return timed(n, nf::narrow64_fwd_name(false, fp), by, fl, s,
                   [&] { return nf::launch_narrow64_fwd(false, fp, s); });
  }
  return run_forward<T>(n, x, nullptr, batch, out, false, s);
}

nf_status check_net(const nf_net* n) {
  if (!n) return fail(NF_EINVAL, "net is NULL");
  return NF_OK;
}

// the entry point's element type must be the net's
template <class T>
nf_status check_net_t(const nf_net* n) {
  nf_status st = check_net(n);
  if (st != NF_OK) return st;
  if (n->dtype != dtype_of<T>())
    return fail(NF_EINVAL, n->dtype == nf::DT_F64
                               ? "the net holds fp64 values: use the _f64 entry points"
                               : "the net holds fp32 values: use the entry points without _f64");
  return NF_OK;
}

nf_status check_train_args(const void* x, const void* y, int64_t batch, double eta,
                           int32_t shards) {
  if (!x || !y) return fail(NF_EINVAL, "x or y is NULL");
  if (batch <= 0) return fail(NF_EINVAL, "batch must be positive");
  if (batch > (int64_t)1 << 30) return fail(NF_ESHAPE, "batch is too large");
  if (shards < 1) return fail(NF_EINVAL, "n_shards must be at least 1");
  if (shards > 65535) return fail(NF_ESHAPE, "n_shards must be at most 65535");
  if (batch % shards != 0) return fail(NF_ESHAPE, "batch must split evenly into n_shards pieces");
  if (!(eta == eta) || eta == __builtin_inf() || eta == -__builtin_inf())
    return fail(NF_EINVAL, "eta must be finite");
  return NF_OK;
}

template <class F>
nf_status guarded(F&& f) {
  try {
    g_err.clear();
    return f();
  } catch (const std::bad_alloc&) {
    return fail(NF_ENOMEM, "host allocation failed");
  } catch (const std::exception& e) {
    return fail(NF_EINVAL, std::string("internal error: ") + e.what());
  } catch (...) {
    return fail(NF_EINVAL, "internal error");
  }
}

nf_status create(const int32_t* dims, int32_t n_dims, const int32_t* acts, int32_t n_acts,
                 int32_t dtype, nf_net** out) {
  if (!out) return fail(NF_EINVAL, "out is NULL");
  if (!dims) return fail(NF_EINVAL, "dims is NULL");
  if (dtype != NF_F32 && dtype != NF_F64) return fail(NF_EINVAL, "unknown dtype");
  if (n_dims < 2) return fail(NF_ESHAPE, "need at least an input and an output layer");
  if (n_dims > 1024) return fail(NF_ESHAPE, "too many layers");
  for (int i = 0; i < n_dims; ++i)
    if (dims[i] < 1 || dims[i] > 65536) return fail(NF_ESHAPE, "layer sizes must be in 1..65536");
  if (n_acts != 0 && n_acts != 1 && n_acts != n_dims - 1)
    return fail(NF_ESHAPE, "n_acts must be 0, 1 or n_dims - 1");
  if (n_acts > 0 && !acts) return fail(NF_EINVAL, "acts is NULL");
  for (int i = 0; i < n_acts; ++i)
    if (acts[i] < NF_GAUSSIAN || acts[i] > NF_TANH) return fail(NF_EINVAL, "unknown activation");

  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return hip_fail(e, "no usable HIP device");
  }
  int ncu = 0;
  e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return hip_fail(e, "hipDeviceGetAttribute");
  }
  nf_net* n = new nf_net();
  n->device = dev;
  n->ncu = ncu;
  n->dtype = dtype == NF_F64 ? nf::DT_F64 : nf::DT_F32;
  n->esz = dtype == NF_F64 ? sizeof(double) : sizeof(float);
  n->dims.assign(dims, dims + n_dims);
  n->layers.resize(n_dims);
  n->narrow = n_dims - 1 <= nf::NARROW_MAX_LAYERS;
  for (int l = 1; l < n_dims; ++l) n->narrow = n->narrow && dims[l] <= nf::NARROW_WIDTH;
  // Narrow nets pad every layer to NARROW_WIDTH rows and the layers after
  // the first to NARROW_WIDTH columns, so their kernels read whole padded
  // blocks without bounds tests; the padding stays zero.
  const int64_t NW = nf::NARROW_WIDTH;
  int64_t off = 0, canon = 0;
  for (int l = 1; l < n_dims; ++l) {
    LayerLayout& ly = n->layers[l];
    ly.in = dims[l - 1];
    ly.out = dims[l];
    ly.act = n_acts == 0 ? NF_SIGMOID : (n_acts == 1 ? acts[0] : acts[l - 1]);
    ly.ldw = (n->narrow && l >= 2) ? NW : round_up(ly.in, 4);
    const int64_t rows = n->narrow ? NW : ly.out;
    ly.w_off = off;
    off = round_up(off + rows * ly.ldw, kAlign);
    ly.b_off = off;
    off = round_up(off + rows, kAlign);
    ly.lda = n->narrow ? NW : round_up(ly.out, 4);
    canon += (int64_t)ly.out * ly.in + ly.out;
  }
  if (n->narrow) {
    n->zero_off = off;
    off = round_up(off + NW * NW + NW, kAlign);
  }
  n->n_params = canon;
  n->dev_elems = off;
  n->actv.assign(n_dims, nullptr);
  n->fbuf.assign(n_dims, nullptr);
  n->dbuf.assign(n_dims, nullptr);
  // both parameter buffers and the tendencies start at zero, padding included
  const size_t bytes = (size_t)off * n->esz;
  e = hipMalloc(&n->pbuf[0], bytes);
  if (e == hipSuccess) e = hipMalloc(&n->pbuf[1], bytes);
  if (e == hipSuccess) e = hipMalloc(&n->grads, bytes);
  if (e == hipSuccess) e = hipMemset(n->pbuf[0], 0, bytes);
  if (e == hipSuccess) e = hipMemset(n->pbuf[1], 0, bytes);
  if (e == hipSuccess) e = hipMemset(n->grads, 0, bytes);
  if (e == hipSuccess && n->narrow && n->dtype == nf::DT_F32) {
    n->w1f_elems = nf::narrow_pack_w1f_elems(dims[0]);
    const size_t pbytes = (size_t)(n->w1f_elems + nf::narrow_pack_w1i_elems(dims[0])) * sizeof(float);
    e = hipMalloc(&n->w1pack, pbytes);
  }
  if (e != hipSuccess) {
    (void)hipGetLastError();
    free_params(n);
    delete n;
    return fail(e == hipErrorOutOfMemory ? NF_ENOMEM : NF_EDEVICE,
                std::string("device allocation failed: ") + hipGetErrorString(e));
  }
  *out = n;
  return NF_OK;
}

// canonical host array <-> device layout (host_src to dev, or dev to host_dst)
nf_status copy_params(nf_net* n, void* dev, const void* host_src, void* host_dst, int64_t count) {
  if (count != n->n_params) return fail(NF_ESHAPE, "parameter count does not match the net");
  DeviceGuard g(n->device);
  if (!g.ok) return fail(NF_EDEVICE, "cannot select the net's device");
  nf_status st = sync_net(n);
  if (st != NF_OK) return st;
  if (host_src) ++n->pver;   // the packed copies of W_1 no longer match
  const size_t es = n->esz;
  char* d = static_cast<char*>(dev);
  int64_t canon = 0;
  for (size_t l = 1; l < n->layers.size(); ++l) {
    const LayerLayout& ly = n->layers[l];
    const size_t wbytes = (size_t)ly.in * es;
    hipError_t e;
    if (host_src) {
      const char* h = static_cast<const char*>(host_src);
      e = hipMemcpy2D(d + ly.w_off * es, ly.ldw * es, h + canon * es, wbytes, wbytes, ly.out,
                      hipMemcpyHostToDevice);
      if (e == hipSuccess)
        e = hipMemcpy(d + ly.b_off * es, h + (canon + (int64_t)ly.out * ly.in) * es,
                      (size_t)ly.out * es, hipMemcpyHostToDevice);
    } else {
      char* h = static_cast<char*>(host_dst);
      e = hipMemcpy2D(h + canon * es, wbytes, d + ly.w_off * es, ly.ldw * es, wbytes, ly.out,
                      hipMemcpyDeviceToHost);
      if (e == hipSuccess)
        e = hipMemcpy(h + (canon + (int64_t)ly.out * ly.in) * es, d + ly.b_off * es,
                      (size_t)ly.out * es, hipMemcpyDeviceToHost);
    }
    if (e != hipSuccess) return hip_fail(e, "parameter copy");
    canon += (int64_t)ly.out * ly.in + ly.out;
  }
  return NF_OK;
}

template <class T>
nf_status set_params(nf_net* net, const T* host_src, int64_t n) {
  return guarded([&]() -> nf_status {
    nf_status st = check_net_t<T>(net);
    if (st != NF_OK) return st;
    if (!host_src) return fail(NF_EINVAL, "host_src is NULL");
    return copy_params(net, net->pbuf[net->cur], host_src, nullptr, n);
  });
}

template <class T>
nf_status get_params(nf_net* net, T* host_dst, int64_t n, bool grads) {
  return guarded([&]() -> nf_status {
    nf_status st = check_net_t<T>(net);
    if (st != NF_OK) return st;
    if (!host_dst) return fail(NF_EINVAL, "host_dst is NULL");
    return copy_params(net, grads ? net->grads : net->pbuf[net->cur], nullptr, host_dst, n);
  });
}

// f'(z_layer) of the last training step's samples, [batch][d_layer] rows
template <class T>
nf_status get_fprime(nf_net* net, int32_t layer, T* host_dst, int64_t batch) {
  return guarded([&]() -> nf_status {
    nf_status st = check_net_t<T>(net);
    if (st != NF_OK) return st;
    if (!host_dst) return fail(NF_EINVAL, "host_dst is NULL");
    const int L = num_layers(net);
    if (layer < 1 || layer >= L) return fail(NF_EINVAL, "layer must be in 1 .. L-1");
    if (net->stash_batch == 0)
      return fail(NF_EINVAL, "the last training step kept f'(z) in registers (or none ran)");
    if (batch != net->stash_batch)
      return fail(NF_ESHAPE, "batch differs from the last training step's");
    DeviceGuard g(net->device);
    if (!g.ok) return fail(NF_EDEVICE, "cannot select the net's device");
    st = sync_net(net);
    if (st != NF_OK) return st;
    const LayerLayout& ly = net->layers[layer];
    const size_t es = net->esz;
    hipError_t e = hipMemcpy2D(host_dst, (size_t)ly.out * es, net->fbuf[layer], (size_t)ly.lda * es,
                               (size_t)ly.out * es, (size_t)batch, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "f' copy");
    return NF_OK;
  });
}

template <class T>
nf_status forward(nf_net* net, const T* d_x, int64_t batch, T* d_out, void* stream) {
  return guarded([&]() -> nf_status {
    nf_status st = check_net_t<T>(net);
    if (st != NF_OK) return st;
    if (!d_x || !d_out) return fail(NF_EINVAL, "x or out is NULL");
    if (batch <= 0) return fail(NF_EINVAL, "batch must be positive");
    if (batch > (int64_t)1 << 30) return fail(NF_ESHAPE, "batch is too large");
    DeviceGuard g(net->device);
    if (!g.ok) return fail(NF_EDEVICE, "cannot select the net's device");
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = infer<T>(net, d_x, batch, d_out, s);
    net->last = s;
    net->used = true;
    return st;
  });
}

template <class T>
nf_status train_batch(nf_net* net, const T* d_x, const T* d_y, int64_t batch, double eta,
                      int32_t n_shards, void* stream) {
  return guarded([&]() -> nf_status {
    nf_status st = check_net_t<T>(net);
    if (st != NF_OK) return st;
    st = check_train_args(d_x, d_y, batch, eta, n_shards);
    if (st != NF_OK) return st;
    DeviceGuard g(net->device);
    if (!g.ok) return fail(NF_EDEVICE, "cannot select the net's device");
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = ensure_ws(net, batch);
    if (st != NF_OK) return st;
    st = train_step<T>(net, d_x, d_y, batch, eta, n_shards, s);
    net->last = s;
    net->used = true;
    return st;
  });
}

// ---------------------------------------------------------------------------
// the training step on the shared scratch array (nf_train_batch_noalloc)
// ---------------------------------------------------------------------------
// The most the piece buffer is asked for by one training step of `batch`
// samples in `shards` shards: the forward pieces (consumed before the
// backward pass starts) or the tendency pieces, whichever is larger.
template <class T>
int64_t partial_need(const nf_net* n, const T* x, int64_t batch, int shards) {
  if (shards == 1 && narrow_rows_ok<T>(n, x)) return 0;
  std::vector<DwPiece> pieces;
  int64_t need = dw_plan(n, batch, shards, &pieces);
  nf::MediumParamsT<T> mp{};
  if (medium_layout<T>(n, batch, &mp)) {
    // the medium path always writes layer 1 as pieces, one or more
    const LayerLayout& l1 = n->layers[1];
    // either kernel may take layer 1, depending on the input rows
    const nf::KSplit ks = fwd_split(n, batch, l1.out, l1.in, false);
    int np = ks.nsplit;
    if (n->dtype == nf::DT_F32 && l1.out <= nf::SKINNY_MAX_UNITS)
      np = std::max(np, fwd_skinny_split(n, batch, l1.out, l1.in).nsplit);
    need = std::max(need, np * round_up(batch * round_up(l1.out, 4), kAlign));
  } else {
    for (int l = 1; l <= num_layers(n); ++l) {
      const LayerLayout& ly = n->layers[l];
      const nf::KSplit ks = fwd_split(n, batch, ly.out, ly.in, true);
      need = std::max(need, fwd_piece_elems(batch, ly.out, ks.nsplit));
    }
  }
  return need;
}

}  // namespace

namespace nf {
// clears n16 16-byte units at p (the workspace's row padding must read as
// zero; a kernel, not hipMemsetAsync, so that the call can be captured)
__global__ void __launch_bounds__(256) zero16_kernel(float4* p, int64_t n16) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += stride)
    p[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}
}  // namespace nf

// The scratch memory of nf_train_batch_noalloc: one array per device, shared
// by every such call on that device.  In host code `scratch` only names the
// symbol; its device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[NF_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

// the device address of the scratch array on device dev, which is current
nf_status scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(NF_EDEVICE, "device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* a = nullptr;
    const hipError_t e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return hip_fail(e, "hipGetSymbolAddress of the scratch array");
    }
    g_scratch_addr[dev] = a;
  }
  *out = g_scratch_addr[dev];
  return NF_OK;
}

// One nf_train_batch step whose per-sample buffers and piece buffer are carved
// out of the scratch array: the net's own workspace is set aside for the call
// and restored after it, and nothing is allocated.
nf_status train_batch_noalloc(nf_net* net, const float* d_x, const float* d_y, int64_t batch,
                              double eta, int32_t n_shards, void* stream) {
  return guarded([&]() -> nf_status {
    nf_status st = check_net_t<float>(net);
    if (st != NF_OK) return st;
    st = check_train_args(d_x, d_y, batch, eta, n_shards);
    if (st != NF_OK) return st;
    DeviceGuard g(net->device);
    if (!g.ok) return fail(NF_EDEVICE, "cannot select the net's device");
    void* base = nullptr;
    st = scratch_address(net->device, &base);
    if (st != NF_OK) return st;
    std::vector<int64_t> aoff, foff, doff;
    const int64_t ws = round_up(ws_layout(net, batch, &aoff, &foff, &doff), kAlign);
    const int64_t part = partial_need<float>(net, d_x, batch, n_shards);
    const double need = (double)(ws + part) * (double)net->esz;
    if (need > (double)NF_NOALLOC_SCRATCH_BYTES)
      return fail(NF_ESHAPE, "this step needs " + std::to_string((int64_t)need) +
                                 " bytes of scratch; nf_train_batch_noalloc has " +
                                 std::to_string((int64_t)NF_NOALLOC_SCRATCH_BYTES));
    hipStream_t s = static_cast<hipStream_t>(stream);
    char* sbase = static_cast<char*>(base);
    // the per-sample buffers' row padding must read as zero, and the array
    // holds whatever the last call left there
    hipError_t e = nf::launch_k(nf::zero16_kernel, dim3(1024), dim3(256), 0, s,
                                reinterpret_cast<float4*>(sbase),
                                ws * (int64_t)net->esz / 16);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return hip_fail(e, "kernel launch");
    }
    // set the net's own buffers aside for the call
    const std::vector<void*> actv = net->actv, fbuf = net->fbuf, dbuf = net->dbuf;
    const int64_t ws_batch = net->ws_batch, partial_elems = net->partial_elems;
    void* partial = net->partial;
    const int prof = net->prof;
    ws_assign(net, sbase, aoff, foff, doff);
    net->ws_batch = batch;
    net->partial = sbase + ws * (int64_t)net->esz;
    net->partial_elems = part;
    net->borrowed = true;
    net->prof = 0;
    st = train_step<float>(net, d_x, d_y, batch, eta, n_shards, s);
    net->actv = actv;
    net->fbuf = fbuf;
    net->dbuf = dbuf;
    net->ws_batch = ws_batch;
    net->partial = partial;
    net->partial_elems = partial_elems;
    net->borrowed = false;
    net->prof = prof;
    net->stash_batch = 0;   // the stash lived in the shared array
    net->last = s;
    net->used = true;
    return st;
  });
}

template <class T>
nf_status train_epoch(nf_net* net, const T* d_x, const T* d_y, int64_t n_samples, int64_t batch,
                      double eta, int32_t n_shards, void* stream) {
  return guarded([&]() -> nf_status {
    nf_status st = check_net_t<T>(net);
    if (st != NF_OK) return st;
    st = check_train_args(d_x, d_y, batch, eta, n_shards);
    if (st != NF_OK) return st;
    if (n_samples <= 0 || n_samples % batch != 0)
      return fail(NF_ESHAPE, "n_samples must be a positive multiple of batch");
    DeviceGuard g(net->device);
    if (!g.ok) return fail(NF_EDEVICE, "cannot select the net's device");
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = ensure_ws(net, batch);
    if (st != NF_OK) return st;
    const int64_t d0 = net->dims.front(), dl = net->dims.back();
    for (int64_t t = 0; t < n_samples / batch; ++t) {
      st = train_step<T>(net, d_x + t * batch * d0, d_y + t * batch * dl, batch, eta, n_shards, s);
      if (st != NF_OK) break;
    }
    net->last = s;
    net->used = true;
    return st;
  });
}

// Windows of the sample set, placed as the example program of section 4
// places its mini-batches: start = int(pos * (n_samples - batch + 1)) with
// the product in the net's element type (the paper's real kind), clamped to
// the last window.
template <class T>
nf_status train_windows(nf_net* net, const T* d_x, const T* d_y, int64_t n_samples, int64_t batch,
                        const T* host_pos, int64_t n_steps, double eta, int32_t n_shards,
                        void* stream) {
  return guarded([&]() -> nf_status {
    nf_status st = check_net_t<T>(net);
    if (st != NF_OK) return st;
    st = check_train_args(d_x, d_y, batch, eta, n_shards);
    if (st != NF_OK) return st;
    if (n_samples < batch) return fail(NF_ESHAPE, "n_samples must be at least batch");
    if (n_steps < 0) return fail(NF_EINVAL, "n_steps must not be negative");
    if (n_steps > 0 && !host_pos) return fail(NF_EINVAL, "host_pos is NULL");
    // every start is checked before anything is launched
    const int64_t last = n_samples - batch;
    const T span = (T)(last + 1);
    std::vector<int64_t> start((size_t)n_steps);
    for (int64_t t = 0; t < n_steps; ++t) {
      const T pos = host_pos[t];
      if (!(pos >= T(0) && pos < T(1))) return fail(NF_EINVAL, "pos values must lie in [0, 1)");
      const T prod = pos * span;
      start[(size_t)t] = std::min((int64_t)prod, last);
    }
    DeviceGuard g(net->device);
    if (!g.ok) return fail(NF_EDEVICE, "cannot select the net's device");
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = ensure_ws(net, batch);
    if (st != NF_OK) return st;
    const int64_t d0 = net->dims.front(), dl = net->dims.back();
    for (int64_t t = 0; t < n_steps && st == NF_OK; ++t)
      st = train_step<T>(net, d_x + start[(size_t)t] * d0, d_y + start[(size_t)t] * dl, batch, eta,
                         n_shards, s);
    net->last = s;
    net->used = true;
    return st;
  });
}

template <class T>
nf_status accuracy(nf_net* net, const T* d_x, const T* d_y, int64_t n, int64_t* host_correct,
                   void* stream) {
  return guarded([&]() -> nf_status {
    nf_status st = check_net_t<T>(net);
    if (st != NF_OK) return st;
    if (!d_x || !d_y || !host_correct) return fail(NF_EINVAL, "x, y or host_correct is NULL");
    if (n <= 0) return fail(NF_EINVAL, "n must be positive");
    if (n > (int64_t)1 << 40) return fail(NF_ESHAPE, "n is too large");
    DeviceGuard g(net->device);
    if (!g.ok) return fail(NF_EDEVICE, "cannot select the net's device");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t d0 = net->dims.front(), dl = net->dims.back();
    // outputs are produced chunk by chunk into a buffer of at most 16 M elements
    const int64_t chunk = std::max<int64_t>(
        1, std::min<int64_t>(n, std::min<int64_t>((int64_t)1 << 14, ((int64_t)1 << 24) / dl)));
    if (chunk * dl > net->eval_elems || !net->dcount) {
      st = sync_net(net);
      if (st != NF_OK) return st;
      if (!net->dcount) {
        hipError_t e = hipMalloc(&net->dcount, sizeof(unsigned long long));
        if (e != hipSuccess) {
          (void)hipGetLastError();
          net->dcount = nullptr;
          return fail(NF_ENOMEM, "hipMalloc of the counter failed");
        }
      }
      if (chunk * dl > net->eval_elems) {
        void* buf = nullptr;
        hipError_t e = hipMalloc(&buf, (size_t)(chunk * dl) * net->esz);
        if (e != hipSuccess) {
          (void)hipGetLastError();
          return fail(NF_ENOMEM, "hipMalloc of the output buffer failed");
        }
        if (net->evalbuf) (void)hipFree(net->evalbuf);
        net->evalbuf = buf;
        net->eval_elems = chunk * dl;
      }
    }
    hipError_t e = hipMemsetAsync(net->dcount, 0, sizeof(unsigned long long), s);
    net->last = s;
    net->used = true;
    if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync");
    T* outb = as<T>(net->evalbuf);
    for (int64_t b = 0; b < n && st == NF_OK; b += chunk) {
      const int64_t m = std::min(chunk, n - b);
      st = infer<T>(net, d_x + b * d0, m, outb, s);
      if (st != NF_OK) break;
      e = nf::launch_count_correct<T>(outb, dl, d_y + b * dl, dl, m, (int)dl, net->dcount, s);
      if (e != hipSuccess) st = hip_fail(e, "count_correct launch");
    }
    if (st != NF_OK) return st;
    unsigned long long count = 0;
    e = hipMemcpyAsync(&count, net->dcount, sizeof(count), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "reading the correct count");
    *host_correct = (int64_t)count;
    return NF_OK;
  });
}

// ---------------------------------------------------------------------------
// save / load: a self-describing little-endian binary file
//   bytes 0..7   magic "NFNET01\n"
//   int32        element type (nf_dtype)
//   int32        n_dims, then int32 dims[n_dims], int32 acts[n_dims - 1]
//   int64        n_params, then n_params elements in canonical order
//   uint64       FNV-1a hash of every byte before it
// ---------------------------------------------------------------------------
constexpr char kMagic[8] = {'N', 'F', 'N', 'E', 'T', '0', '1', '\n'};

struct Fnv {
  uint64_t h = 1469598103934665603ull;
  void add(const void* p, size_t n) {
    const unsigned char* b = static_cast<const unsigned char*>(p);
    for (size_t i = 0; i < n; ++i) {
      h ^= b[i];
      h *= 1099511628211ull;
    }
  }
};

struct File {
  FILE* f = nullptr;
  ~File() {
    if (f) std::fclose(f);
  }
};

bool little_endian() {
  const uint32_t one = 1;
  unsigned char c;
  std::memcpy(&c, &one, 1);
  return c == 1;
}

nf_status save(nf_net* net, const char* path) {
  if (!path) return fail(NF_EINVAL, "path is NULL");
  if (!little_endian()) return fail(NF_EINVAL, "the file format is little-endian");
  std::vector<char> params((size_t)net->n_params * net->esz);
  nf_status st = copy_params(net, net->pbuf[net->cur], nullptr, params.data(), net->n_params);
  if (st != NF_OK) return st;
  std::vector<char> out;
  auto put = [&](const void* p, size_t n) {
    out.insert(out.end(), static_cast<const char*>(p), static_cast<const char*>(p) + n);
  };
  const int32_t dtype = net->dtype == nf::DT_F64 ? NF_F64 : NF_F32;
  const int32_t nd = (int32_t)net->dims.size();
  put(kMagic, sizeof(kMagic));
  put(&dtype, 4);
  put(&nd, 4);
  for (int32_t d : net->dims) put(&d, 4);
  for (size_t l = 1; l < net->layers.size(); ++l) {
    const int32_t a = net->layers[l].act;
    put(&a, 4);
  }
  const int64_t np = net->n_params;
  put(&np, 8);
  put(params.data(), params.size());
  Fnv h;
  h.add(out.data(), out.size());
  put(&h.h, 8);
  File f;
  f.f = std::fopen(path, "wb");
  if (!f.f) return fail(NF_EINVAL, std::string("cannot open ") + path + " for writing");
  if (std::fwrite(out.data(), 1, out.size(), f.f) != out.size() || std::fflush(f.f) != 0)
    return fail(NF_EINVAL, std::string("cannot write ") + path);
  return NF_OK;
}

nf_status load(const char* path, nf_net** out) {
  if (!path || !out) return fail(NF_EINVAL, "path or out is NULL");
  if (!little_endian()) return fail(NF_EINVAL, "the file format is little-endian");
  File f;
  f.f = std::fopen(path, "rb");
  if (!f.f) return fail(NF_EINVAL, std::string("cannot open ") + path);
  std::vector<char> buf;
  char chunk[1 << 16];
  size_t got;
  while ((got = std::fread(chunk, 1, sizeof(chunk), f.f)) > 0) {
    buf.insert(buf.end(), chunk, chunk + got);
    if (buf.size() > ((size_t)1 << 36)) return fail(NF_EINVAL, "file too large");
  }
  size_t pos = 0;
  auto take = [&](void* dst, size_t n) {
    if (buf.size() < pos + n) return false;
    std::memcpy(dst, buf.data() + pos, n);
    pos += n;
    return true;
  };
  const std::string bad = std::string("not a valid network file: ") + path;
  char magic[8];
  int32_t dtype = 0, nd = 0;
  if (!take(magic, 8) || std::memcmp(magic, kMagic, 8) != 0) return fail(NF_EINVAL, bad);
  if (!take(&dtype, 4) || !take(&nd, 4)) return fail(NF_EINVAL, bad);
  if (dtype != NF_F32 && dtype != NF_F64) return fail(NF_EINVAL, bad + " (element type)");
  if (nd < 2 || nd > 1024) return fail(NF_EINVAL, bad + " (layer count)");
  std::vector<int32_t> dims(nd), acts(nd - 1);
  for (auto& d : dims)
    if (!take(&d, 4)) return fail(NF_EINVAL, bad);
  for (auto& a : acts)
    if (!take(&a, 4)) return fail(NF_EINVAL, bad);
  int64_t np = 0;
  if (!take(&np, 8)) return fail(NF_EINVAL, bad);
  int64_t want = 0;
  for (int l = 1; l < nd; ++l) {
    if (dims[l - 1] < 1 || dims[l - 1] > 65536 || dims[l] < 1 || dims[l] > 65536)
      return fail(NF_EINVAL, bad + " (layer sizes)");
    want += (int64_t)dims[l] * dims[l - 1] + dims[l];
  }
  const size_t es = dtype == NF_F64 ? sizeof(double) : sizeof(float);
  if (np != want) return fail(NF_EINVAL, bad + " (parameter count)");
  if (buf.size() != pos + (size_t)np * es + 8) return fail(NF_EINVAL, bad + " (length)");
  Fnv h;
  h.add(buf.data(), pos + (size_t)np * es);
  uint64_t stored = 0;
  std::memcpy(&stored, buf.data() + pos + (size_t)np * es, 8);
  if (stored != h.h) return fail(NF_EINVAL, bad + " (checksum)");
  nf_net* n = nullptr;
  nf_status st = create(dims.data(), nd, acts.data(), nd - 1, dtype, &n);
  if (st != NF_OK) return st;
  st = copy_params(n, n->pbuf[n->cur], buf.data() + pos, nullptr, np);
  if (st != NF_OK) {
    const std::string msg = g_err;
    free_params(n);
    delete n;
    return fail(st, msg);
  }
  *out = n;
  return NF_OK;
}

}  // namespace

extern "C" {

nf_status nf_save(nf_net* net, const char* path) {
  return guarded([&]() -> nf_status {
    nf_status st = check_net(net);
    return st != NF_OK ? st : save(net, path);
  });
}

nf_status nf_load(const char* path, nf_net** out) {
  return guarded([&]() { return load(path, out); });
}

nf_status nf_net_create(const int32_t* dims, int32_t n_dims, const int32_t* acts, int32_t n_acts,
                        nf_net** out) {
  return guarded([&]() { return create(dims, n_dims, acts, n_acts, NF_F32, out); });
}

nf_status nf_net_create_ex(const int32_t* dims, int32_t n_dims, const int32_t* acts,
                           int32_t n_acts, int32_t dtype, nf_net** out) {
  return guarded([&]() { return create(dims, n_dims, acts, n_acts, dtype, out); });
}

int32_t nf_net_dtype(const nf_net* net) {
  if (!net) return -1;
  return net->dtype == nf::DT_F64 ? NF_F64 : NF_F32;
}

nf_status nf_net_destroy(nf_net* net) {
  return guarded([&]() -> nf_status {
    if (!net) return NF_OK;
    DeviceGuard g(net->device);
    nf_status st = sync_net(net);
    clear_recs(net);
    free_ws(net);
    if (net->partial) (void)hipFree(net->partial);
    if (net->evalbuf) (void)hipFree(net->evalbuf);
    if (net->dcount) (void)hipFree(net->dcount);
    free_params(net);
    delete net;
    return st;
  });
}

int64_t nf_param_count(const nf_net* net) { return net ? net->n_params : -1; }

nf_status nf_set_params(nf_net* net, const float* host_src, int64_t n) {
  return set_params<float>(net, host_src, n);
}
nf_status nf_get_params(nf_net* net, float* host_dst, int64_t n) {
  return get_params<float>(net, host_dst, n, false);
}
nf_status nf_get_grads(nf_net* net, float* host_dst, int64_t n) {
  return get_params<float>(net, host_dst, n, true);
}
nf_status nf_forward(nf_net* net, const float* d_x, int64_t batch, float* d_out, void* stream) {
  return forward<float>(net, d_x, batch, d_out, stream);
}
nf_status nf_train_batch(nf_net* net, const float* d_x, const float* d_y, int64_t batch, float eta,
                         int32_t n_shards, void* stream) {
  return train_batch<float>(net, d_x, d_y, batch, (double)eta, n_shards, stream);
}
nf_status nf_train_batch_noalloc(nf_net* net, const float* d_x, const float* d_y, int64_t batch,
                                 float eta, int32_t n_shards, void* stream) {
  return train_batch_noalloc(net, d_x, d_y, batch, eta, n_shards, stream);
}
nf_status nf_train_epoch(nf_net* net, const float* d_x, const float* d_y, int64_t n_samples,
                         int64_t batch, float eta, int32_t n_shards, void* stream) {
  return train_epoch<float>(net, d_x, d_y, n_samples, batch, (double)eta, n_shards, stream);
}
nf_status nf_train_single(nf_net* net, const float* d_x, const float* d_y, float eta,
                          void* stream) {
  return train_batch<float>(net, d_x, d_y, 1, (double)eta, 1, stream);
}
nf_status nf_train_windows(nf_net* net, const float* d_x, const float* d_y, int64_t n_samples,
                           int64_t batch, const float* host_pos, int64_t n_steps, float eta,
                           int32_t n_shards, void* stream) {
  return train_windows<float>(net, d_x, d_y, n_samples, batch, host_pos, n_steps, (double)eta,
                              n_shards, stream);
}
nf_status nf_accuracy(nf_net* net, const float* d_x, const float* d_y, int64_t n,
                      int64_t* host_correct, void* stream) {
  return accuracy<float>(net, d_x, d_y, n, host_correct, stream);
}

nf_status nf_set_params_f64(nf_net* net, const double* host_src, int64_t n) {
  return set_params<double>(net, host_src, n);
}
nf_status nf_get_params_f64(nf_net* net, double* host_dst, int64_t n) {
  return get_params<double>(net, host_dst, n, false);
}
nf_status nf_get_grads_f64(nf_net* net, double* host_dst, int64_t n) {
  return get_params<double>(net, host_dst, n, true);
}
nf_status nf_get_fprime(nf_net* net, int32_t layer, float* host_dst, int64_t batch) {
  return get_fprime<float>(net, layer, host_dst, batch);
}
nf_status nf_get_fprime_f64(nf_net* net, int32_t layer, double* host_dst, int64_t batch) {
  return get_fprime<double>(net, layer, host_dst, batch);
}
nf_status nf_forward_f64(nf_net* net, const double* d_x, int64_t batch, double* d_out,
                         void* stream) {
  return forward<double>(net, d_x, batch, d_out, stream);
}
nf_status nf_train_batch_f64(nf_net* net, const double* d_x, const double* d_y, int64_t batch,
                             double eta, int32_t n_shards, void* stream) {
  return train_batch<double>(net, d_x, d_y, batch, eta, n_shards, stream);
}
nf_status nf_train_epoch_f64(nf_net* net, const double* d_x, const double* d_y, int64_t n_samples,
                             int64_t batch, double eta, int32_t n_shards, void* stream) {
  return train_epoch<double>(net, d_x, d_y, n_samples, batch, eta, n_shards, stream);
}
nf_status nf_train_single_f64(nf_net* net, const double* d_x, const double* d_y, double eta,
                              void* stream) {
  return train_batch<double>(net, d_x, d_y, 1, eta, 1, stream);
}
nf_status nf_train_windows_f64(nf_net* net, const double* d_x, const double* d_y,
                               int64_t n_samples, int64_t batch, const double* host_pos,
                               int64_t n_steps, double eta, int32_t n_shards, void* stream) {
  return train_windows<double>(net, d_x, d_y, n_samples, batch, host_pos, n_steps, eta, n_shards,
                               stream);
}
nf_status nf_accuracy_f64(nf_net* net, const double* d_x, const double* d_y, int64_t n,
                          int64_t* host_correct, void* stream) {
  return accuracy<double>(net, d_x, d_y, n, host_correct, stream);
}

nf_status nf_profile(nf_net* net, int32_t repeats) {
  return guarded([&]() -> nf_status {
    nf_status st = check_net(net);
    if (st != NF_OK) return st;
    DeviceGuard g(net->device);
    if (repeats < 0 || repeats > 1000) return fail(NF_EINVAL, "repeats must be in 0..1000");
    if (repeats) {
      st = sync_net(net);
      if (st != NF_OK) return st;
      clear_recs(net);
    }
    net->prof = repeats;
    return NF_OK;
  });
}

nf_status nf_profile_read(nf_net* net, nf_kernel_stat* out, int32_t cap, int32_t* count) {
  return guarded([&]() -> nf_status {
    nf_status st = check_net(net);
    if (st != NF_OK) return st;
    if (!count || (cap > 0 && !out)) return fail(NF_EINVAL, "out or count is NULL");
    if (cap < 0) return fail(NF_EINVAL, "cap must not be negative");
    DeviceGuard g(net->device);
    st = sync_net(net);
    if (st != NF_OK) return st;
    std::vector<nf_kernel_stat> agg;
    for (const auto& r : net->recs) {
      float ms = 0.0f;
      hipError_t e = hipEventElapsedTime(&ms, r.a, r.b);
      if (e != hipSuccess) {
        clear_recs(net);
        return hip_fail(e, "hipEventElapsedTime");
      }
      nf_kernel_stat* k = nullptr;
      for (auto& a : agg)
        if (std::strncmp(a.name, r.name, sizeof(a.name)) == 0) k = &a;
      if (!k) {
        agg.push_back(nf_kernel_stat{});
        k = &agg.back();
        std::snprintf(k->name, sizeof(k->name), "%s", r.name);
      }
      const double one = ms / (r.repeats > 1 ? r.repeats : 1);
      k->min_ms = k->launches == 0 ? one : std::min(k->min_ms, one);
      k->max_ms = k->launches == 0 ? one : std::max(k->max_ms, one);
      k->launches += 1;
      k->total_ms += one;
      k->bytes += r.bytes;
      k->flops += r.flops;
    }
    clear_recs(net);
    std::sort(agg.begin(), agg.end(),
              [](const nf_kernel_stat& a, const nf_kernel_stat& b) {
                return a.total_ms > b.total_ms;
              });
    const int32_t n = (int32_t)std::min<size_t>(agg.size(), (size_t)cap);
    for (int32_t i = 0; i < n; ++i) out[i] = agg[i];
    *count = n;
    return NF_OK;
  });
}

const char* nf_last_error(void) { return g_err.c_str(); }

}  // extern "C"
