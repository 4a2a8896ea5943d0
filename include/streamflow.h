/*
 * streamflow.h - C ABI of the stream-batched rectified-flow step on MI355X (gfx950).
 *
 * The method (StreamFlow, arXiv 2511.22009) keeps a queue of in-flight latents,
 * each at its own denoising time, and advances all of them with ONE velocity-network
 * call per step (Sec. 3.2, Eq. 5), followed by a per-sample Euler update
 * x' = x + (t_next - t) v (Sec. 3.1.1 discretization; Alg. 1, its final update) and a
 * shift of the queue: fresh noise enters at slot 0 and the oldest latent leaves
 * finished (Sec. 3.4.1-3.4.2; Alg. 2).
 *
 * The velocity network is a DiT-style adaLN transformer that outputs v directly; its
 * shape comes from the weight blob. Every computation step runs in HIP kernels on the
 * GPU; the host side only validates arguments and enqueues launches.
 *
 * Conventions shared by every call:
 *   - Latents x, velocities v, z_new and x_done are DEVICE pointers to fp32 NCHW data,
 *     one latent = C*H*W floats, slots contiguous: x[B][C][H][W].
 *   - t[] and dt[] are HOST arrays of B floats. They are copied into kernel arguments
 *     at call time and not retained.
 *   - Slot 0 is the newest latent (largest t), slot B-1 the oldest (Alg. 2's order:
 *     the batch is [z_new, buffer] and the finished sample is the last entry).
 *   - Calls enqueue work on `hip_stream` (a hipStream_t; NULL = the default stream) and
 *     return without waiting. One handle is used by one host thread at a time.
 *   - Every call returns SF_OK (0) or a negative SF_E_* code. All argument and blob
 *     validation happens on the host before any HIP call, so a rejected call has no
 *     effect. A HIP failure (allocation, launch, or an earlier asynchronous fault seen
 *     by the launch check) returns SF_E_HIP. Nothing aborts the process.
 *   - The caller owns every device buffer it passes; the library never frees or keeps
 *     them. The library owns the weights and workspace inside the handle.
 */
#ifndef STREAMFLOW_H
#define STREAMFLOW_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sf_model sf_model;

/* Status codes. */
enum {
  SF_OK = 0,
  SF_E_INVAL = -1,        /* bad argument (null pointer, size out of range, non-finite t/dt) */
  SF_E_BLOB = -2,         /* weight blob malformed (magic, version, shape fields, byte count) */
  SF_E_NOTLOADED = -3,    /* handle is NULL where a loaded model is required */
  SF_E_OOM = -4,          /* device allocation failed */
  SF_E_HIP = -5,          /* a HIP runtime call or kernel launch failed */
  SF_E_UNSUPPORTED = -6   /* valid blob, but a shape this build has no kernel for */
};

/* Arithmetic modes. BF16: bf16 weights and GEMM/attention operands with fp32
 * accumulation, fp32 residual stream, latents and velocities. FP32: fp32 throughout. */
enum { SF_PREC_BF16 = 0, SF_PREC_FP32 = 1 };

/* Largest number of network rows one call may run (latents, doubled under guidance). */
#define SF_MAX_ROWS 64

/* Conditioning for networks with cross-attention (the conditioning c of Alg. 2's
 * network call, and its ApplyCFG / HandleCFG steps).
 *   ctx      device fp32 [B][ctx_len][ctx_dim]: the context of each slot's latent.
 *   null_ctx device fp32 [ctx_len][ctx_dim]: the unconditional context shared by every
 *            unconditional row, or NULL for no guidance.
 *   guidance w: with null_ctx set, the network runs 2B rows (B with ctx, then B with
 *            null_ctx, each at its slot's t) and v = v_u + w (v_c - v_u). */
typedef struct sf_cond {
  const float* ctx;
  const float* null_ctx;
  float guidance;
} sf_cond;

/* Shape and mode of a loaded model. */
typedef struct sf_info {
  int C, H, W, p, D, L, heads, mlp, tdim, ctx_len, ctx_dim, has_cross;
  int tokens;            /* N = (H/p) * (W/p) tokens per latent */
  int mod_width;         /* L*6*D + 2*D: width of one row of the adaLN table */
  int precision;         /* SF_PREC_* */
  int max_rows;
  size_t weight_bytes;   /* device bytes held for weights */
  size_t workspace_bytes;/* device bytes held for activations */
  int vt_ld;             /* row length (keys) of the transposed-v buffer SF_BUF_VT, a multiple of 64 */
  int vt_key_perm;       /* 1 (bf16 mode): key t of SF_BUF_VT sits at column (t with bits 2
                            and 3 swapped), the layout the bf16 attention reads; 0: column t */
} sf_info;

/* Parse a weight blob, upload the weights (converted to bf16 in SF_PREC_BF16 mode) and
 * size the workspace for up to `max_rows` network rows (1..SF_MAX_ROWS).
 *
 * Blob layout (little-endian): 64-byte header = magic "SFW1", u32 version (1), u32
 * C,H,W,p,D,L,heads,mlp,tdim,ctx_len,ctx_dim,has_cross, u64 seed; then fp32 tensors:
 * W_pe[D][p*p*C], b_pe[D], pos[N][D], W_t1[D][tdim], b_t1[D], W_t2[D][D], b_t2[D];
 * per block W_mod[6D][D], b_mod[6D], W_qkv[3D][D], b_qkv[3D], W_o[D][D], b_o[D],
 * (if has_cross) W_qx[D][D], b_qx[D], W_kvx[2D][ctx_dim], b_kvx[2D], W_ox[D][D],
 * b_ox[D], then W_fc1[mlp][D], b_fc1[mlp], W_fc2[D][mlp], b_fc2[D]; finally
 * W_fmod[2D][D], b_fmod[2D], W_f[p*p*C][D], b_f[p*p*C]. Linear weights are [out][in].
 * The byte count must match exactly.
 *
 * `blob` is a HOST pointer; it is read during the call and not retained. On success
 * *out owns device memory until sf_free. Errors: SF_E_INVAL (null blob/out, bad
 * precision or max_rows), SF_E_BLOB, SF_E_UNSUPPORTED (head dim not a multiple of 8
 * or above 128, a width not a multiple of 8, H or W not a multiple of p; in bf16 mode
 * an activation of max_rows rows reaching 2^31 bytes, e.g. max_rows x tokens x the MLP
 * width x 2, since the bf16 kernels use 32-bit byte offsets), SF_E_OOM, SF_E_HIP. No
 * handle is returned on failure. The environment variable SF_FAIL_ALLOC_AFTER=n makes
 * the (n+1)-th device allocation of a load fail, to exercise the SF_E_OOM path. */
int sf_load_weights(const void* blob, size_t nbytes, int precision, int max_rows, sf_model** out);

/* Release everything the handle owns. NULL is a no-op. Waits for the device. */
void sf_free(sf_model* m);

/* Text for a status code (static storage). */
const char* sf_strerror(int code);

/* Copy the model's shape and mode into *info. */
int sf_get_info(const sf_model* m, sf_info* info);

/* The heterogeneous-timestep network call (Sec. 3.2, Eq. 5): v[k] = v_theta(x[k], t[k])
 * for k < B, every slot at its own t. x: device [B][C][H][W]; t: host [B] in [0, 1]
 * (the network sees 1000 t); v: device [B][C][H][W] output. cond: NULL for an
 * unconditioned network; required when the network has cross-attention (see sf_cond).
 * Rows run = B, or 2B with guidance; must be <= max_rows. */
int sf_velocity(sf_model* m, const float* x, const float* t, int B, const sf_cond* cond,
                float* v, void* hip_stream);

/* One stream step (Eq. 5 network call, then Alg. 1's per-sample Euler update, then
 * Alg. 2's shift), in place on x:
 *   v = v_theta(x[0:B], t[0:B]);  x'_k = x_k + dt_k v_k   (dt signed: t_next - t)
 *   x_done != NULL (full pipeline): x_done <- x'_{B-1}; x[k+1] <- x'_k for k < B-1;
 *                                   x[0] <- z_new. The queue keeps B slots.
 *   x_done == NULL (filling):       x[k+1] <- x'_k for k < B; x[0] <- z_new. The queue
 *                                   grows to B+1 slots, so x must hold B+1 latents.
 * z_new (device, one latent) is required. The Euler product and sum are rounded
 * separately (no fused multiply-add), the same as a plain fp32 x + dt * v. */
int sf_stream_step(sf_model* m, float* x, const float* t, const float* dt, int B,
                   const sf_cond* cond, const float* z_new, float* x_done, void* hip_stream);

/* The Euler update and shift of sf_stream_step alone, on a caller-supplied velocity
 * v: device [B][C][H][W]. Same in-place semantics and rounding. */
int sf_euler_shift(sf_model* m, float* x, const float* v, const float* dt, int B,
                   const float* z_new, float* x_done, void* hip_stream);

/* The per-sample timestep conditioning alone: for each k < B, the sinusoidal embedding
 * of 1000 t[k], the timestep MLP, and every adaLN projection. table: device fp32
 * [B][mod_width]; row k holds, for each block, (shift1, scale1, gate1, shift2, scale2,
 * gate2) of width D each, then the final layer's (shift, scale). */
int sf_modulation(sf_model* m, const float* t, int B, float* table, void* hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): sf_modulation with its two
 * intermediates (the timestep MLP's hidden layer and SiLU(c), [B][D] fp32 each) in a
 * fixed device array of the library (1 MiB per GPU, allocated with the library's code
 * object and held until the process ends) instead of the model's workspace. Same
 * arguments and results as sf_modulation (bit-identical table); B may be 1..SF_MAX_ROWS
 * regardless of max_rows (SF_E_INVAL beyond: the array holds 2 x 64 x 2048 floats).
 * Calls no allocating routine. Every call on one GPU uses that GPU's one array, so
 * calls that overlap on a GPU (on different streams, or from different models on the
 * same GPU) race on it; calls in stream order on one stream do not. */
int sf_modulation_noalloc(sf_model* m, const float* t, int B, float* table, void* hip_stream);

/* Test hook: run the network on B rows (cond as in sf_velocity) through the patch
 * embedding and the first `blocks` blocks (0..L) and copy the fp32 residual stream to
 * h: device [rows][N][D]. */
int sf_residual(sf_model* m, const float* x, const float* t, int B, const sf_cond* cond,
                int blocks, float* h, void* hip_stream);

/* Internal buffers readable through sf_debug_read. After a network call (sf_velocity,
 * sf_stream_step or sf_residual) they hold what that call left, i.e. the intermediates
 * of the LAST block it ran. Element type: fp32 for SF_BUF_H and SF_BUF_TABLE; the
 * compute type (bf16 in SF_PREC_BF16 mode, else fp32) for the others.
 *   SF_BUF_H     [rows][N][D]           residual stream
 *   SF_BUF_ACT   [rows][N][D]           last LayerNorm + modulate output (the MLP input)
 *   SF_BUF_Q/K   [rows][heads][N][dh]   self-attention queries / keys
 *   SF_BUF_VT    [rows][heads][dh][ldv] self-attention values, transposed; ldv = N
 *                                       rounded up to a multiple of 64 (sf_info.vt_ld),
 *                                       keys permuted when sf_info.vt_key_perm is 1
 *   SF_BUF_ATTN  [rows][N][D]           attention output before the output projection
 *   SF_BUF_MLP   [rows][N][mlp]         GELU(fc1) output
 *   SF_BUF_TABLE [B][mod_width]         adaLN table (rows k < B) */
enum { SF_BUF_H = 0, SF_BUF_ACT, SF_BUF_Q, SF_BUF_K, SF_BUF_VT, SF_BUF_ATTN, SF_BUF_MLP, SF_BUF_TABLE };

/* Test hook: copy the first `bytes` bytes of internal buffer `buffer` to device memory
 * `dst` (enqueued on hip_stream). SF_E_INVAL if bytes exceeds the buffer. */
int sf_debug_read(sf_model* m, int buffer, void* dst, size_t bytes, void* hip_stream);

/* Test hook: the model's self-attention (Sec. 3.2's network, one layer's
 * softmax(q k^T / sqrt(dh)) v per row and head) on caller buffers, in the layouts and
 * element type of the internal buffers above: q, k device [rows][heads][N][dh], vT device
 * [rows][heads][dh][vt_ld] (keys permuted when vt_key_perm is 1, columns past N zero),
 * o device [rows][N][D] output. rows 1..SF_MAX_ROWS (independent of max_rows). The
 * same kernels as the network call for that many rows. */
int sf_attention(sf_model* m, const void* q, const void* k, const void* vT, void* o, int rows, void* hip_stream);

/* Kernel classes for event timing. */
enum {
  SF_KC_TEMB = 0,   /* timestep embedding, MLP and adaLN projections */
  SF_KC_EMBED,      /* patchify + patch embed + position table */
  SF_KC_LN,         /* LayerNorm + adaLN modulate */
  SF_KC_QKV,        /* QKV projection GEMM */
  SF_KC_ATTN,       /* self-attention */
  SF_KC_PROJ,       /* attention output projection GEMM + gated residual */
  SF_KC_FC1,        /* MLP up-projection GEMM + GELU */
  SF_KC_FC2,        /* MLP down-projection GEMM + gated residual */
  SF_KC_CROSS,      /* every cross-attention kernel */
  SF_KC_HEAD,       /* final LayerNorm + modulate + linear + unpatchify */
  SF_KC_EULER,      /* guidance combine, Euler update and queue shift */
  SF_KC_COUNT
};

/* The latent an image-to-image run admits: the point of the straight path between a
 * reference latent and noise at the schedule's first time t0 (Sec. 2 straight paths;
 * t = 1 is noise): out = (1 - t0) x_ref + t0 z, products and sum rounded to fp32
 * separately. x_ref, z, out: device [C][H][W]; out may alias z or x_ref (element-wise).
 * t0 in [0, 1]. Pass `out` as z_new of sf_stream_step with a schedule starting at t0. */
int sf_noise_latent(sf_model* m, const float* x_ref, const float* z, float t0, float* out, void* hip_stream);

/* PeRFlow time windows (Sec. 2 time-window mechanism; Sec. 3.3 vectorized window lookup
 * and batch parameters; Alg. 1). With a scheduler set, the network output of
 * sf_stream_step is read as a noise prediction eps and each slot's update is
 *   X_pred = lambda_t x + eta_t eps;  v = (X_pred - x) / (t^e - t);  x' = x + dt v
 * with the window of t found as k = #{j < windows : t > j / windows + eps} (at least 1),
 * running from t^s = k / windows down to t^e = (k - 1) / windows,
 * gamma = sqrt(abar(t^s) / abar(t^e)), lambda_s = 1 / gamma,
 * eta_s = -sqrt(1 - gamma^2) / gamma, denom = lambda_s (t - t^s) + (t^e - t),
 * lambda_t = lambda_s (t^e - t^s) / denom, eta_t = eta_s (t^e - t) / denom.
 * t is normalised time in [0, 1] (1 = noise) and dt is signed. abar is alphas_cumprod of
 * the scaled-linear schedule (beta on a linear grid in sqrt(beta) from beta_start to
 * beta_end over train_steps steps), read at index round(u (train_steps - 1)). The
 * per-slot coefficients are computed in fp64 on the GPU; x' = A x + B eps in fp32.
 * Guidance, when present, combines the two noise predictions as it combines velocities. */
typedef struct {
  int windows;        /* number of equal windows over [0, 1], 1..4096 */
  int train_steps;    /* length of the schedule, 2..1048576 (1000 for the latent diffusion models) */
  float beta_start;   /* 0 < beta_start < beta_end < 1 (0.00085, 0.012) */
  float beta_end;
  double eps;         /* window lookup tolerance, 0 <= eps < 1 / windows (1e-6) */
} sf_perflow;

/* Set (p != NULL) or clear (p == NULL: Euler on the velocity, the default) the
 * scheduler of sf_stream_step and sf_scheduler_shift. Synchronous: builds the schedule
 * on the host in fp64 and uploads it (one device allocation, kept until sf_free).
 * Drops cached graphs. SF_E_INVAL on out-of-range fields. On SF_E_OOM or SF_E_HIP the
 * scheduler is cleared (Euler on the velocity), never left half set. The schedule's
 * allocation fails when SF_FAIL_ALLOC_AFTER is 0, to exercise that path. */
int sf_set_scheduler(sf_model* m, const sf_perflow* p);

/* The update and shift of sf_stream_step alone, with the model's scheduler, for a
 * given network output `out` [B][C][H][W] (a velocity without a scheduler, a noise
 * prediction with one). t and dt are host [B]. Test hook and building block. */
int sf_scheduler_shift(sf_model* m, float* x, const float* out, const float* t, const float* dt, int B,
                       const float* z_new, float* x_done, void* hip_stream);

/* Graph replay of the step (Sec. 3.5 asks for static execution of heterogeneous steps;
 * here t is data, so one captured launch sequence serves every mix of timesteps).
 * While enabled, sf_velocity and sf_stream_step capture their launches on the caller's
 * stream into a HIP graph the first time a given call (entry point, pointers, B, t, dt,
 * conditioning) is seen, and replay that graph on every identical later call. Up to 64
 * graphs are kept (least recently used goes first). Requires a non-null stream (the
 * legacy default stream cannot be captured); on the null stream, or while any kernel
 * class is being timed, calls run eagerly. Results are bit-identical to eager calls.
 * Disabling destroys the cached graphs. The captured sequences contain kernel launches
 * only (no memset or copy nodes). Returns SF_E_HIP if a capture or instantiation fails
 * (the call's work is then not enqueued). */
int sf_graph_enable(sf_model* m, int enable);
/* Number of graphs currently cached and number of replays served from the cache. */
int sf_graph_stats(const sf_model* m, int* cached, long* replays);

/* Modulation cache (the per-sample conditioning computed once while the timesteps stay
 * the same). The adaLN table of a call depends on its timesteps only (Eq. 5: each
 * sample's own t enters the network through the timestep embedding, Sec. 3.2), and in
 * the steady state of a fixed schedule every queue slot sees the same t at every step
 * (Alg. 2). While enabled, sf_velocity and sf_stream_step skip the conditioning launches
 * (timestep MLP and adaLN projections) when the previous network call on the same stream
 * computed the table for exactly the same t[0..B) (bitwise); results are bit-identical
 * to calls without the cache. Off by default. Enabling or disabling forgets the cached
 * state; a failed call invalidates it. The cache assumes stream order: a call on another
 * stream never hits it. Returns SF_E_NOTLOADED for a null model. */
int sf_modulation_cache(sf_model* m, int enable);
/* Number of network calls that reused the cached table (skips counted at enqueue). */
int sf_modulation_cache_stats(const sf_model* m, long* skips);

/* Context reuse for cross-attention (Alg. 2: the conditioning c of each latent stays
 * with it while it moves through the queue, and ApplyCFG / HandleCFG pair every latent
 * with the one unconditional context). The keys and values of a context depend on the
 * context and the weights only. Every network call keeps them per context ENTRY for all
 * blocks at once: the B conditional rows use the entries of their own contexts and all
 * unconditional rows share the entry of null_ctx (computed once per call, not per row).
 * While enabled, entries also outlive the call: each slot's context is compared, bitwise
 * and on the GPU, with the context of the entry that slot used in the previous call and
 * with that of the entry of the slot before it (where the shift of sf_stream_step moved
 * it), likewise the null context; an equal one is reused and only the others are
 * projected. Results are bit-identical to calls without reuse. The entries live in the
 * model's workspace and are updated in stream order, so calls that use the cache must
 * run in order on one stream. Off by default. Enabling or disabling forgets every entry
 * and waits for the device; a failed call forgets them too. A no-op (SF_OK) for networks
 * without cross-attention. Returns SF_E_NOTLOADED for a null model, SF_E_HIP on a HIP
 * failure. */
int sf_context_cache(sf_model* m, int enable);
/* Calls that went through the entry lookup while enabled, and the context entries they
 * projected (the rest were reused). Waits for the device. Zero for networks without
 * cross-attention. */
int sf_context_cache_stats(const sf_model* m, long* calls, long* projected);

/* Test and bench hook: while enabled, every launch of kernel class `kc` is timed by a
 * pair of HIP events. For a class that is one kernel the events are attached to that
 * kernel's dispatch (its own start and end); SF_KC_TEMB and SF_KC_CROSS, which launch
 * several kernels, are bracketed by events recorded on the launch stream. At most 4096
 * launches per class are recorded; later ones are counted but not timed. sf_timing_read
 * waits for the recorded events, returns the summed milliseconds and the number of
 * timed launches, and clears the record. */
int sf_timing_enable(sf_model* m, int kc, int enable);
int sf_timing_read(sf_model* m, int kc, double* total_ms, long* launches);

#ifdef __cplusplus
}
#endif

#endif /* STREAMFLOW_H */
