/*
 * nf.h - C ABI of the MI355X (gfx950) library for mini-batch training of
 * fully connected feed-forward networks, after Curcic, "A parallel Fortran
 * framework for neural networks and deep learning" (arXiv:1902.06714).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Real data is IEEE fp32, the paper's default real32 kind (section 3.1), or
 *   IEEE fp64, its real64 kind, chosen per net at creation (nf_net_create_ex).
 *   The entry points without a suffix take fp32 data and serve fp32 nets;
 *   their _f64 twins take fp64 data and serve fp64 nets.  Calling one family on
 *   a net of the other precision returns NF_EINVAL.
 * - Batches are row-major: a batch of B samples of width d is B rows of d
 *   contiguous floats, sample after sample.  This is byte-identical to the
 *   paper's column-major x(d, B) (section 3.4, batch training).
 * - Canonical parameter order: for l = 1..L (L = n_dims - 1 layers after the
 *   input), the weights W_l as a row-major [d_l][d_{l-1}] array (row j holds
 *   the weights from every unit of layer l-1 into unit j of layer l), then the
 *   biases b_l[d_l].  The paper stores w(this, next) column-major on the
 *   source layer (section 3.1, layer definition), which has the same bytes.
 *   The paper's unused input-layer biases and last-layer weights are not
 *   stored.  The device layout is private; get/set convert.
 * - Pointers named d_* are device pointers on the net's device; pointers named
 *   host_* are host memory.  The caller owns all of them; the library never
 *   frees or retains them past the call.
 * - `stream` is a hipStream_t passed as void* (NULL means the default stream).
 *   Compute calls only enqueue work on that stream and return; the caller
 *   keeps the inputs alive and unmodified until the stream reaches that work.
 * - Every call returns an nf_status.  On error nothing has been enqueued, the
 *   net is unchanged, and nf_last_error() gives a message for this thread.
 *   No C++ exception crosses the ABI.
 * - A net is not thread-safe: calls on one net must not overlap.
 */
#ifndef NF_H
#define NF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Opaque network: owned by the library, created by nf_net_create. */
typedef struct nf_net nf_net;

/* The activation functions of section 2 (Gaussian, RELU, sigmoid, step,
 * tangent hyperbolic).  f and its derivative f' (taken at the stored
 * pre-activation z, section 3.3):
 *   NF_GAUSSIAN  exp(-z^2)            -2 z exp(-z^2)
 *   NF_RELU      max(0, z)            1 if z > 0 else 0
 *   NF_SIGMOID   1 / (1 + exp(-z))    sigma(z) sigma(-z)   (section 3.1)
 *   NF_STEP      1 if z > 0 else 0    0
 *   NF_TANH      tanh(z)              1 - tanh(z)^2                         */
typedef enum {
  NF_GAUSSIAN = 0,
  NF_RELU = 1,
  NF_SIGMOID = 2,
  NF_STEP = 3,
  NF_TANH = 4
} nf_act;

/* Element type of a net's parameters and data (section 3.1: the real kind is
 * chosen when the library is built, real32 by default). */
typedef enum {
  NF_F32 = 0,
  NF_F64 = 1
} nf_dtype;

typedef enum {
  NF_OK = 0,
  NF_EINVAL = -1,  /* bad argument: NULL pointer, bad enum, count <= 0 ...   */
  NF_ESHAPE = -2,  /* sizes that do not fit the net or each other           */
  NF_ENOMEM = -3,  /* device or host allocation failed                      */
  NF_EDEVICE = -4  /* a HIP runtime call failed (includes "no GPU")         */
} nf_status;

/* Create a network (the network constructor of section 3.1).
 * dims[0..n_dims-1]: units per layer including input and output layers,
 *   n_dims >= 2, every entry in 1 .. 65536.
 * acts[0..n_acts-1]: nf_act values.  n_acts = 0: sigmoid on every layer (the
 *   paper's default); n_acts = 1: that activation on every layer (the paper's
 *   case); n_acts = n_dims - 1: one per layer after the input.
 * The net lives on the HIP device current at the call.  Its parameters start
 * at zero: load them with nf_set_params (the single-GPU stand-in for the
 * broadcast of initial parameters, section 3.5).
 * *out receives the handle; it is set only on success. */
nf_status nf_net_create(const int32_t* dims, int32_t n_dims, const int32_t* acts,
                        int32_t n_acts, nf_net** out);

/* nf_net_create with a choice of element type: dtype is an nf_dtype.  An
 * NF_F64 net keeps its parameters, tendencies and per-sample buffers in fp64
 * and computes in fp64 (the real64 kind of section 3.1); it is driven with
 * the _f64 entry points below. */
nf_status nf_net_create_ex(const int32_t* dims, int32_t n_dims, const int32_t* acts,
                           int32_t n_acts, int32_t dtype, nf_net** out);

/* The nf_dtype of a net, or -1 for NULL. */
int32_t nf_net_dtype(const nf_net* net);

/* Destroy a network; waits for its outstanding work.  NULL is a no-op. */
nf_status nf_net_destroy(nf_net* net);

/* Number of elements in the canonical parameter vector:
 * sum over l of d_l * d_{l-1} + d_l.  Returns -1 for NULL. */
int64_t nf_param_count(const nf_net* net);

/* Copy n = nf_param_count(net) floats in canonical order from host memory
 * into the net.  Waits for the net's outstanding work first; returns after
 * the copy is complete. */
nf_status nf_set_params(nf_net* net, const float* host_src, int64_t n);

/* Copy the current parameters, canonical order, into host memory (n floats).
 * Waits for the net's outstanding work. */
nf_status nf_get_params(nf_net* net, float* host_dst, int64_t n);

/* Copy the tendencies of the most recent nf_train_batch step (the weight and
 * bias gradients of the quadratic cost summed over the whole mini-batch,
 * before scaling by eta/B; section 3.3-3.5) into host memory, canonical order,
 * n floats.  Zero before the first step.  Waits for outstanding work. */
nf_status nf_get_grads(nf_net* net, float* host_dst, int64_t n);

/* Copy f'(z_layer), the activation derivative at the pre-activations of layer
 * `layer` (1 .. L-1) that the most recent training step kept for
 * back-propagation (section 3.2: z is stored for the backward pass), into
 * host memory as [batch][d_layer] rows, batch = that step's batch.  For a relu
 * layer the entries are its kink decisions, 1 where z > 0 and 0 elsewhere:
 * a parity check takes them to resolve units that lie within rounding of the
 * kink, where either side is a correct result.  Only steps that store f' in
 * device memory keep it: NF_EINVAL after a step that held f' in registers
 * (nets of at most 32 units per layer after the input with one shard, or at
 * most 128 units in 2 to 4 layers), before any step, and once a larger batch
 * has replaced the per-sample buffers; NF_ESHAPE if batch differs from the
 * step's.  Waits for the net's outstanding work. */
nf_status nf_get_fprime(nf_net* net, int32_t layer, float* host_dst, int64_t batch);

/* Batched inference: the network output for every sample, storing nothing in
 * the net (the output function of section 3.2).
 * d_x: [batch][d_0] input, d_out: [batch][d_L] output; batch >= 1. */
nf_status nf_forward(nf_net* net, const float* d_x, int64_t batch, float* d_out,
                     void* stream);

/* One SGD step on one mini-batch (sections 3.2-3.5):
 * forward propagation of every sample, the output delta
 * (a_L - y) f'(z_L), the hidden deltas (W_{l+1}^T delta_{l+1}) f'(z_l) with
 * the weights from before this step, the weight and bias tendencies summed
 * over the batch, and W_l -= (eta / batch) * sum, b_l -= (eta / batch) * sum.
 * n_shards >= 1 splits the batch into that many equal contiguous pieces
 * whose tendencies are formed separately and added in piece order (the
 * collective sum of section 3.5, on one GPU); batch % n_shards must be 0.
 * d_x: [batch][d_0] inputs, d_y: [batch][d_L] targets (one-hot for
 * classification). */
nf_status nf_train_batch(nf_net* net, const float* d_x, const float* d_y, int64_t batch,
                         float eta, int32_t n_shards, void* stream);

/* nf_train_batch for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * The same step, bit for bit, with the per-sample buffers and the tendency
 * pieces placed in a scratch array that the library holds on each device
 * (NF_NOALLOC_SCRATCH_BYTES, a device variable of the library: the runtime
 * maps it with the library's code on that device, and it stays until the
 * process ends) instead of the net's own workspace; the call allocates
 * nothing (no hipMalloc or hipFree, no memset node: the array is cleared by
 * a kernel) and leaves the net's own workspace as it was.  fp32 nets only.
 * Errors as nf_train_batch, plus NF_ESHAPE (nothing enqueued, the net
 * unchanged) when the step needs more than NF_NOALLOC_SCRATCH_BYTES: about
 * 3 * batch * (sum of the layer widths, each rounded up to 4; 32 for
 * networks of at most 32 units per layer) floats of per-sample buffers, plus
 * the tendency pieces of sharded or split batches.  Every such call on a
 * device uses the same array and starts by clearing what it needs: calls
 * that can overlap on one device (different streams, or threads) race and
 * must be ordered by the caller.  The step's f'(z) is not kept afterwards
 * (nf_get_fprime reports none), and nf_profile recording is suspended for
 * the call. */
#define NF_NOALLOC_SCRATCH_BYTES (48 << 20)
nf_status nf_train_batch_noalloc(nf_net* net, const float* d_x, const float* d_y, int64_t batch,
                                 float eta, int32_t n_shards, void* stream);

/* Consecutive mini-batches: samples [t*batch, (t+1)*batch) for
 * t = 0 .. n_samples/batch - 1, one nf_train_batch step each, in order
 * (the epoch loop of section 4 without the random window).  n_samples must be
 * a positive multiple of batch. */
nf_status nf_train_epoch(nf_net* net, const float* d_x, const float* d_y, int64_t n_samples,
                         int64_t batch, float eta, int32_t n_shards, void* stream);

/* One training step on a single sample (section 3.4, train_single): the
 * forward pass, back-propagation and the update for the sample d_x [d_0] with
 * target d_y [d_L].  Identical to nf_train_batch with batch 1 and one shard. */
nf_status nf_train_single(nf_net* net, const float* d_x, const float* d_y, float eta, void* stream);

/* Training on randomly placed windows of the sample set, as the paper's
 * example program draws its mini-batches (section 4): for t = 0 .. n_steps-1,
 * in order, one nf_train_batch step on samples [s_t, s_t + batch) with
 *     s_t = min(int(pos[t] * (n_samples - batch + 1)), n_samples - batch),
 * the product taken in fp32 (the paper's default real kind) and truncated.
 * Windows may overlap and samples may be left out, as in the paper.  The
 * uniform numbers pos[0 .. n_steps-1] in [0, 1) are drawn by the caller and
 * passed in host memory; NF_EINVAL if one is outside [0, 1) or not finite
 * (nothing is launched then).  d_x: [n_samples][d_0], d_y: [n_samples][d_L]. */
nf_status nf_train_windows(nf_net* net, const float* d_x, const float* d_y, int64_t n_samples,
                           int64_t batch, const float* host_pos, int64_t n_steps, float eta,
                           int32_t n_shards, void* stream);

/* Classification accuracy (section 4): the number of the n samples whose
 * network output and target have their largest entry at the same index (the
 * first index among equal largest entries, as Fortran's maxloc).  d_x: [n][d_0]
 * inputs, d_y: [n][d_L] targets (one-hot class vectors in the paper).  A
 * sample whose output or target holds a NaN counts as incorrect.  Runs on
 * `stream`, waits for it, and writes the count to *host_correct. */
nf_status nf_accuracy(nf_net* net, const float* d_x, const float* d_y, int64_t n,
                      int64_t* host_correct, void* stream);

/* The fp64 twins of the calls above, for nets created with dtype NF_F64: the
 * same operations, arguments and errors, with every real array (parameters,
 * tendencies, inputs, targets, outputs, window positions) in fp64 and eta in
 * fp64.  nf_train_windows_f64 forms pos * (n_samples - batch + 1) in fp64. */
nf_status nf_set_params_f64(nf_net* net, const double* host_src, int64_t n);
nf_status nf_get_params_f64(nf_net* net, double* host_dst, int64_t n);
nf_status nf_get_grads_f64(nf_net* net, double* host_dst, int64_t n);
nf_status nf_get_fprime_f64(nf_net* net, int32_t layer, double* host_dst, int64_t batch);
nf_status nf_forward_f64(nf_net* net, const double* d_x, int64_t batch, double* d_out,
                         void* stream);
nf_status nf_train_batch_f64(nf_net* net, const double* d_x, const double* d_y, int64_t batch,
                             double eta, int32_t n_shards, void* stream);
nf_status nf_train_epoch_f64(nf_net* net, const double* d_x, const double* d_y, int64_t n_samples,
                             int64_t batch, double eta, int32_t n_shards, void* stream);
nf_status nf_train_single_f64(nf_net* net, const double* d_x, const double* d_y, double eta,
                              void* stream);
nf_status nf_train_windows_f64(nf_net* net, const double* d_x, const double* d_y,
                               int64_t n_samples, int64_t batch, const double* host_pos,
                               int64_t n_steps, double eta, int32_t n_shards, void* stream);
nf_status nf_accuracy_f64(nf_net* net, const double* d_x, const double* d_y, int64_t n,
                          int64_t* host_correct, void* stream);

/* Save a network to a file and create one from it (section 2 lists saving
 * and loading networks among the framework's features; the paper does not
 * fix a format).  The file is little-endian binary:
 *   bytes 0..7  "NFNET01\n"
 *   int32       element type (nf_dtype)
 *   int32       n_dims, then int32 dims[n_dims] and int32 acts[n_dims - 1]
 *   int64       n_params, then the parameters in canonical order, in the
 *               net's element type
 *   uint64      FNV-1a 64-bit hash of every preceding byte
 * nf_save waits for the net's outstanding work.  nf_load checks the whole file
 * (magic, sizes, length, hash) before it creates the net on the current
 * device; a file that fails a check gives NF_EINVAL and *out is not written.
 * Tendencies and per-sample buffers are not saved. */
nf_status nf_save(nf_net* net, const char* path);
nf_status nf_load(const char* path, nf_net** out);

/* Per-kernel timing, for measuring the method's computational performance the
 * way section 5 reports it (elapsed time), one kernel at a time.  While
 * recording is on, every kernel the net launches is timed with a pair of HIP
 * events, and the library notes the algorithmic bytes the kernel must move
 * (inputs read once, outputs written once) and the flops of its contraction
 * (2 per multiply-add, no padding). */
typedef struct {
  char name[64];      /* kernel family, e.g. "gemm_fwd_stash_128x128" */
  int64_t launches;   /* launches recorded since the last read             */
  double total_ms;    /* sum of the measured durations (ms)                */
  double bytes;       /* algorithmic bytes, summed over the launches       */
  double flops;       /* algorithmic flops, summed over the launches       */
  double min_ms;      /* shortest and longest single measured duration (ms) */
  double max_ms;
} nf_kernel_stat;

/* repeats = 0 turns recording off.  repeats = 1 turns it on (discarding
 * anything recorded and not yet read) with the two events of a launch bound
 * to that kernel's dispatch, so each launch is charged its own start-to-end
 * time and nothing is added between launches.  repeats = R >= 2 instead runs
 * each launch R times in a row between two events recorded on its stream and
 * charges it the average of the R runs; repeating is harmless because no
 * kernel writes a buffer it reads (a training step reads the parameters from
 * one buffer and writes the updated ones to another), but the repeats find
 * their inputs in cache.  repeats must be in 0 .. 1000. */
nf_status nf_profile(nf_net* net, int32_t repeats);

/* Wait for the recorded work, then write one entry per kernel name (at most
 * cap entries, ordered by total time, largest first) to out[] and their number
 * to *count; the records are then cleared. */
nf_status nf_profile_read(nf_net* net, nf_kernel_stat* out, int32_t cap, int32_t* count);

/* Measurement aids: the device's own peaks, against which the roofline
 * fractions of the kernels above are read (the published peaks are quoted
 * beside them).  Each runs one kernel on `stream` (void* hipStream_t), waits
 * for it, and returns the kernel's own start-to-end time in *host_ms.
 * nf_calib_read: a streaming read of `bytes` bytes at d_src (a positive
 * multiple of 16 at a 16-byte aligned device address), 4 workgroups of 256
 * threads per compute unit, 16-byte loads; d_sink is device scratch of at
 * least NF_CALIB_SINK_BYTES bytes.
 * nf_calib_copy: the same access pattern copying d_src to d_dst.
 * nf_calib_mfma: a loop of independent matrix-core instructions, `iters`
 * (rounded up to a multiple of 8) rounds of 8 per wave on 2 (fp32) or 4
 * (fp64) workgroups of 4 waves per compute unit
 * (v_mfma_f32_32x32x2f32 for dtype NF_F32, v_mfma_f64_16x16x4f64 for
 * NF_F64); *host_flops receives the flops it performed (2 per multiply-add)
 * and *host_clock_ghz the mean shader clock of its waves, from the shader
 * cycle counter against the 100 MHz constant clock.  d_sink as above.
 * Errors: NF_EINVAL for NULL pointers, bad sizes or alignment; NF_EDEVICE
 * when there is no device or a HIP call fails. */
/* nf_calib_spin: enqueue on `stream` one kernel that returns after `us`
 * microseconds (0 .. 1e6; one wave polling the 100 MHz constant clock) and
 * return at once.  Work the host enqueues behind it meanwhile starts back to
 * back when it ends, so kernels timed with nf_profile(net, 1), whose launches
 * cost the host more than their run time, still run as in an untimed
 * sequence. */
#define NF_CALIB_SINK_BYTES (1 << 20)
nf_status nf_calib_spin(void* stream, double us);
nf_status nf_calib_read(const void* d_src, int64_t bytes, void* d_sink, void* stream,
                        double* host_ms);
nf_status nf_calib_copy(void* d_dst, const void* d_src, int64_t bytes, void* stream,
                        double* host_ms);
nf_status nf_calib_mfma(int32_t dtype, int64_t iters, void* d_sink, void* stream,
                        double* host_ms, double* host_flops, double* host_clock_ghz);

/* Message for the last failed call on this thread ("" if none).  The pointer
 * stays valid until the next nf_* call on the same thread. */
const char* nf_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* NF_H */
