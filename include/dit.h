/*
 * dit.h -- C ABI of the MI355X (gfx950) Diffusion-Transformer step library.
 *
 * The library computes one denoising step of an MMDiT-class Diffusion
 * Transformer, the unit of work that TetriServe (arXiv 2510.01565) schedules:
 * section 4.1 states the serving problem as executing the denoising steps of
 * requests, each at its own output resolution, and section 2.2 / Table 1 fixes
 * the image-token count of a request, (resolution/16)^2.  The step consists of
 * adaLN-modulated LayerNorm, a QKV projection with 2-D rotary embedding of the
 * image tokens, joint text+image attention, a GELU MLP with gated residuals,
 * the final adaLN layer that predicts the flow-matching velocity, and the Euler
 * update x' = x - dt*v.  Everything runs as HIP kernels on the caller's stream.
 *
 * Conventions shared by every call
 *  - All tensors are device memory owned by the caller, dense and row-major.
 *    Element types: DIT_BF16 = bfloat16 (raw 16-bit storage), DIT_F32 = float.
 *  - No call allocates or frees device memory and none synchronises the host;
 *    all work is enqueued on `stream` (a hipStream_t; NULL = default stream)
 *    and the call returns before it finishes.  Buffers must stay valid until
 *    the enqueued work completes.
 *  - Arguments are validated on the host before anything is enqueued; an
 *    invalid call returns an error code and enqueues nothing.
 *  - Every call returns a dit_status.  On failure dit_last_error() returns a
 *    message, kept per calling thread until that thread's next call.
 *  - A packed batch concatenates requests in order.  Hidden states inside the
 *    library and in dit_block_forward use the "stream-major" row order: first
 *    the text tokens of every request (request 0's, then request 1's, ...),
 *    then the image tokens of every request in the same order.  Image tokens
 *    of a request are its latent patches in row-major grid order (token p sits
 *    at grid row p / grid_w, column p % grid_w).
 *  - Linear weights use the [out, in] layout; all weights and biases of a
 *    model have the config's dtype.
 */
#ifndef DIT_H
#define DIT_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DIT_OK = 0,
  DIT_ERR_INVALID_ARG = 1, /* null pointer, bad size or shape, inconsistent batch */
  DIT_ERR_UNSUPPORTED = 2, /* valid request this build does not implement (head_dim, dtype, sizes) */
  DIT_ERR_WORKSPACE = 3,   /* workspace pointer null or smaller than dit_workspace_size() */
  DIT_ERR_HIP = 4          /* a HIP runtime call or kernel launch failed */
} dit_status;

typedef enum { DIT_F32 = 0, DIT_BF16 = 1 } dit_dtype;

/* Largest number of requests in one packed batch. */
#define DIT_MAX_REQUESTS 16
/* Largest image grid side (tokens per axis); 256 = a 4096 px image. */
#define DIT_MAX_GRID 256

/*
 * Model shape.  Blocks: n_double double-stream blocks (text and image keep
 * their own weights, attention is joint) followed by n_single single-stream
 * blocks (one weight set over the joint sequence).  tie_streams != 0 gives the
 * double blocks one weight set for both streams (a plain joint adaLN block).
 * Fixed readings: LayerNorm eps = ln_eps, biased variance, no affine; adaLN
 * LN(x)*(1+scale)+shift; GELU tanh form; RoPE splits head_dim in two halves
 * (grid row, grid column) with consecutive-pair rotation and base rope_theta.
 * dtype is the storage type of weights, latents, text embeddings and the
 * velocity: DIT_BF16 computes with bf16 operands and fp32 accumulation, an
 * fp32 residual stream, fp32 LayerNorm statistics and fp32 softmax state;
 * DIT_F32 computes everything in fp32 with no reduced-precision arithmetic.
 */
typedef struct {
  int hidden;        /* H, a multiple of 64 */
  int heads;         /* heads * head_dim == hidden */
  int head_dim;      /* bf16: 128 or 64; f32: 64 */
  int mlp_ratio;     /* MLP width = mlp_ratio * hidden */
  int n_double;
  int n_single;
  int in_channels;   /* C_in of the patchified latents, a multiple of 8 */
  int text_dim;      /* width of the text embeddings, a multiple of 8 */
  int time_freq_dim; /* width of the sinusoidal timestep embedding, a multiple of 8, at most 4096 */
  int tie_streams;
  float rope_theta;
  float ln_eps;
  int dtype;         /* dit_dtype */
  int flags;         /* DIT_FLAG_* bits, 0 for the defaults */
} dit_config;

/*
 * DIT_FLAG_BATCH_INVARIANT: every output bit of a request is independent of
 * what it is packed with.  Without it, a bf16 GEMM launch with too few output
 * tiles to fill the GPU may split its K range over several blocks whose fp32
 * partial sums are added in a fixed order, and a bf16 attention launch whose
 * last round of 128-query tiles is at most a quarter full may split those tiles'
 * key ranges (head dim 128, requests of one length); results stay bitwise
 * identical from run to run, but the order of the sums (and so the last bits)
 * can change with the batch composition.  The flag also removes the split's
 * workspace.
 */
#define DIT_FLAG_BATCH_INVARIANT 1

/*
 * A packed batch of n_req requests (1..DIT_MAX_REQUESTS).  All arrays are
 * host memory of n_req entries, read during the call only.  Request r has
 * grid_h[r] * grid_w[r] image tokens (1 <= grid side <= DIT_MAX_GRID) and
 * n_txt[r] >= 0 text tokens; t[r] is its timestep in [0, 1] (may be NULL
 * where a call does not use it).
 */
typedef struct {
  int n_req;
  const int* grid_h;
  const int* grid_w;
  const int* n_txt;
  const float* t;
} dit_batch;

/* Device pointers to every parameter, in manifest order (dit_weight_manifest). */
typedef struct {
  const void* const* tensors; /* host array of n_tensors device pointers */
  int n_tensors;
} dit_weights;

/* Number of parameter tensors of a model (the DiT backbone of section 2.1,
 * at the shapes of the models of section 6.1). */
dit_status dit_weight_count(const dit_config* cfg, int* count);

/*
 * Name and shape of parameter `index` (0 <= index < count): the parameters of
 * the Diffusion Transformer that each denoising step runs (section 2.1, "DiT
 * Background"; the served models of section 6.1).  The paper fixes no layout;
 * this one is the library's own.  *name points to
 * a library-owned string valid until the library is unloaded; shape[0..ndim)
 * receives the dimensions ([out, in] for a weight, [n] for a bias).  The
 * adaLN modulation weights of all blocks are one tensor "mod.w" [rows, H] /
 * "mod.b" [rows]: per double block its image stream's 6H rows then (unless
 * tied) its text stream's 6H rows, then 3H rows per single block, then the
 * final layer's 2H rows; chunks are (shift1, scale1, gate1, shift2, scale2,
 * gate2), (shift, scale, gate) and (shift, scale).
 */
dit_status dit_weight_manifest(const dit_config* cfg, int index, const char** name, int shape[2], int* ndim);

/*
 * Bytes of device workspace that dit_step / dit_block_forward need for this
 * batch.  They grow with its token count: (resolution / 16)^2 image tokens per
 * request (section 2.2, Table 1) plus its text tokens.  The workspace holds
 * activations, Q / K / V^T, the modulation vectors and, for bf16 models
 * without DIT_FLAG_BATCH_INVARIANT, 96 MiB of split-K partial sums and 4 KiB
 * of counters (zeroed by the calls themselves; no initialisation needed).
 */
dit_status dit_workspace_size(const dit_config* cfg, const dit_batch* batch, size_t* bytes);

/*
 * One velocity prediction for every request of the batch (TetriServe
 * section 4.1: one denoising step of each request; section 2.2: its token
 * count).  latents: [sum_r grid_h*grid_w, in_channels] in config dtype,
 * requests concatenated; text_emb: [sum_r n_txt, text_dim] in config dtype;
 * velocity: output, same shape and dtype as latents.  batch->t is required.
 * ws: device workspace of at least dit_workspace_size() bytes, 256-byte
 * aligned; its contents are scratch.
 */
dit_status dit_step(const dit_config* cfg, const dit_weights* w, const dit_batch* batch,
                    const void* latents, const void* text_emb, void* velocity,
                    void* ws, size_t ws_bytes, void* stream);

/*
 * dit_step without a workspace argument, for callers that cannot allocate
 * device memory: code under HIP graph capture, serving loops that forbid
 * allocation.  Same inputs, outputs, kernels and results as dit_step; the
 * workspace is a static area of DIT_NOALLOC_SCRATCH_BYTES inside the library,
 * one per GPU, held from the first use of the library on that GPU until the
 * process ends.  A batch whose dit_workspace_size() exceeds that returns
 * DIT_ERR_WORKSPACE before anything is enqueued.  The call allocates nothing
 * (its first call on a GPU looks up that GPU's scratch address).  All calls on
 * one GPU share its scratch and each call overwrites it: calls that overlap
 * on one GPU (concurrent streams, or a second call enqueued on another stream
 * before the first finishes) race and give wrong results.
 */
#define DIT_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)
dit_status dit_step_noalloc(const dit_config* cfg, const dit_weights* w, const dit_batch* batch,
                            const void* latents, const void* text_emb, void* velocity, void* stream);

/*
 * One transformer block of the denoising network, in place (section 2.1: the
 * step is a stack of transformer blocks whose attention spans the whole token
 * sequence; a sequence-parallel group computes each block together).
 * kind 0 = double-stream block `index`
 * (0 <= index < n_double), kind 1 = single-stream block `index`.
 * hidden: fp32 [sum_r n_txt + sum_r grid_h*grid_w, hidden] in stream-major
 * order, read and overwritten.  cond: fp32 device [n_req, hidden], the
 * conditioning vector c of each request (the modulation input, before SiLU).
 * The text and image rows travel in this one fp32 buffer rather than as two
 * separate tensors: the residual stream stays fp32 between blocks, the
 * single-stream blocks work on the joint sequence, and a double block's text
 * and image rows are then two contiguous row ranges of the same buffer, so no
 * concatenation or split is needed between block kinds.
 */
dit_status dit_block_forward(const dit_config* cfg, const dit_weights* w, int kind, int index,
                             const dit_batch* batch, float* hidden, const float* cond,
                             void* ws, size_t ws_bytes, void* stream);

/*
 * The latent update that ends a denoising step and produces the input of the
 * request's next step (section 4.1: a request is a chain of dependent steps;
 * section 5, "Latent Transfer": the latents are what passes between steps).
 * Flow-matching Euler update x <- x - dt[r] * v for every request, computed in
 * fp32 and rounded once to `dtype`.  latents (in/out) and velocity:
 * [sum_r grid_h*grid_w, channels] of type dtype; dt: host array [n_req].
 */
dit_status euler_update(const dit_batch* batch, int channels, int dtype, void* latents,
                        const void* velocity, const float* dt, void* stream);

/*
 * Joint attention alone, O = softmax(Q K^T / sqrt(head_dim)) V per head and
 * per request over the request's sequence [text; image] (no mask inside a
 * request, nothing across requests).  Sequence order here is the joint order:
 * request 0's n_txt[0] text then grid_h[0]*grid_w[0] image tokens, then
 * request 1's, ...  q, k, v, o: [T_joint, heads, head_dim] of type dtype
 * (head h of token p at (p*heads + h)*head_dim).  This is the call a
 * sequence-parallel rank makes on the heads it owns after the all-to-all
 * (section 2.1, Ulysses attention: tokens and heads are transposed across
 * GPUs before local attention).
 * head_dim: 128 or 64 for DIT_BF16 (bf16 operands, fp32 softmax state and
 * accumulation, P rounded to bf16 for P V), 64 for DIT_F32 (all fp32);
 * anything else returns DIT_ERR_UNSUPPORTED before any launch.
 * ws: at least dit_attention_workspace_size() bytes: V^T, plus for DIT_BF16
 * at head_dim 128, when the last round of 128-query tiles (two per CU) is at
 * most a quarter full after two or more full rounds and every request has one
 * length, the fp32 partial results of those tiles' key ranges (up to 33 MiB),
 * merged in a fixed order (bitwise repeatable).
 */
dit_status dit_attention_workspace_size(const dit_batch* batch, int heads, int head_dim, int dtype,
                                        size_t* bytes);
dit_status dit_attention(const dit_batch* batch, int heads, int head_dim, int dtype, const void* q,
                         const void* k, const void* v, void* o, void* ws, size_t ws_bytes, void* stream);

/*
 * Plain GEMM of the library's kernels: Y[M, N] = X[M, K] W[N, K]^T + b[N]
 * with bf16 operands and fp32 accumulation, Y stored as fp32 (out_dtype =
 * DIT_F32) or bf16 (DIT_BF16).  b may be NULL.  dtype DIT_F32 takes fp32 X, W,
 * b and computes in fp32.  K must be a multiple of 8 and every row 16-byte
 * aligned.  Exposed so that each kernel can be checked on its own; it
 * implements no passage of the paper by itself.
 */
dit_status dit_linear(int M, int N, int K, int dtype, const void* x, const void* w, const void* b,
                      void* y, int out_dtype, void* stream);

/*
 * Kernel timing for measurement.  dit_profile_start() makes every later call
 * (from any thread) bracket each kernel launch with a pair of HIP events on
 * the launch's own stream, grouped by kernel family ("gemm_bf16_256x128",
 * "attention_bf16", "ln_modulate", ...), together with the launch's
 * algorithmic FLOPs and HBM bytes.  dit_profile_stop() waits for those events,
 * sums them per family, turns recording off and returns the number of
 * families; dit_profile_entry() reads family i (name valid until the next
 * dit_profile_start).  Timing adds two event records per launch, so measure
 * throughput with profiling off.  Not meant for concurrent use.
 */
dit_status dit_profile_start(void);
dit_status dit_profile_stop(int* n_families);
dit_status dit_profile_entry(int i, const char** family, long* launches, double* total_ms, double* flops,
                             double* bytes);

/* Message of the last failed call on this thread ("" if none). */
const char* dit_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* DIT_H */
