/*
 * kvd.h -- C ABI of libkvd, the MI355X (gfx950) library for KV-Direct's hot
 * path: recompute attention keys and values from checkpointed residual-stream
 * vectors, then run grouped-query decode attention over them.
 *
 * The operations follow the paper's statement of the problem:
 *   - RMSNorm, Sec. 3.1, Eqs. (rmsnorm), (rms_def);
 *   - the per-head projections, Sec. 3.1, Eqs. (q_proj), (k_proj), (v_proj);
 *   - RoPE, Sec. 3.2, Eqs. (rope_cos), (rope_sin);
 *   - the reconstruction identity, Sec. 3.2, Eqs. (k_recon), (v_recon);
 *   - attention, Sec. 3.1, Eqs. (attn_weights), (head_output);
 *   - one KV-Direct decode step, Sec. 3.4, Algorithm 1 (RECOMPUTE_KV, CONCAT,
 *     ATTENTION) at cache budget 0, optionally with a stored tail of keys.
 *
 * Conventions shared by every call
 * --------------------------------
 * Memory.   Every tensor pointer is a DEVICE pointer, owned by the caller and
 *           aligned to 16 bytes.  The library never allocates, frees or
 *           synchronises: each call validates its arguments on the host,
 *           enqueues its kernels on `stream` (a hipStream_t; NULL means the
 *           null stream) and returns.  Outputs must not alias inputs.
 * Dtype.    shape->dtype (KVD_F32 or KVD_BF16) is the element type of every
 *           tensor a call reads or writes, except `pos*` (int32) and the
 *           workspace (opaque).  Arithmetic accumulates in fp32; K, V and q are
 *           rounded once (round-to-nearest-even) to the dtype after RoPE.
 * Layouts.  Row-major, innermost index last:
 *             residuals  h      [B][h_ld][d_model]   rows 0..T-1 of each sequence used
 *             gamma             [d_model]
 *             W_q               [n_q_heads  * head_dim][d_model]   ([out][in])
 *             W_k, W_v          [n_kv_heads * head_dim][d_model]   ([out][in])
 *             q, attention out  [B][n_q_heads][head_dim]
 *             K/V store         [B][n_kv_heads][t_cap][head_dim]   (kvd_kv_view)
 *           Weights are stored [out][in], the transpose of the paper's
 *           row-vector W (h W), so head h owns rows h*head_dim ..
 *           (h+1)*head_dim-1.  shape->w_layout selects how each weight matrix
 *           is laid out in memory: KVD_W_ROWMAJOR (as above), KVD_W_PACKED
 *           (the MFMA operand order written by kvd_pack_weights; bf16 only),
 *           both holding the same values and giving bit-identical results, or
 *           KVD_W_PACKED_GAMMA (kvd_pack_weights_gamma: gamma folded into the
 *           packed weights; gamma arguments are then not read).
 * Norm.     hbar = h / sqrt(mean(h^2) + rms_eps) * gamma.
 * RoPE.     Consecutive pairs (2i, 2i+1), 0-based, are rotated by
 *           +p * rope_theta^(-2i/head_dim), p the token's absolute position.
 * GQA.      Query head h reads KV head h / (n_q_heads / n_kv_heads).
 * Scale.    Scores are q.k / sqrt(head_dim); softmax subtracts the maximum.
 * Positions pos0[b] (int32, device): residual row t of sequence b sits at
 *           absolute position pos0[b] + t.
 * Errors.   Validation happens before any HIP call and returns a status; no
 *           call aborts or throws.  KVD_ERR_DEVICE reports a failed launch.
 *           kvd_last_error() returns a thread-local description of the last
 *           non-OK status on the calling thread.
 */
#ifndef KVD_H
#define KVD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVD_ABI_VERSION 8

typedef enum {
  KVD_OK = 0,
  KVD_ERR_NULL = 1,         /* a required pointer is NULL */
  KVD_ERR_SHAPE = 2,        /* inconsistent or out-of-range sizes */
  KVD_ERR_UNSUPPORTED = 3,  /* valid arguments the library has no kernel for */
  KVD_ERR_WORKSPACE = 4,    /* workspace NULL or smaller than required */
  KVD_ERR_ALIGN = 5,        /* a tensor pointer is not 16-byte aligned */
  KVD_ERR_DEVICE = 6        /* the HIP runtime reported an error */
} kvd_status;

typedef enum { KVD_F32 = 0, KVD_BF16 = 1 } kvd_dtype;

/* Memory layout of W_q / W_k / W_v (see kvd_pack_weights).
 * KVD_W_PACKED_GAMMA: packed by kvd_pack_weights_gamma, with the RMSNorm weight
 * folded in (W diag(gamma), an exact identity of Eqs. rmsnorm / k_proj: the
 * norm's scale moves from the residual to the weights' columns).  The kernels
 * then stage the residuals unchanged and do not read gamma (calls accept NULL
 * for it).  K/V and q produced from folded weights differ from the other
 * layouts' by rounding only; every producer of this layout (recompute,
 * prefill, the current token's projection, the fused kernels) gives
 * bit-identical values for the same residuals.                               */
typedef enum { KVD_W_ROWMAJOR = 0, KVD_W_PACKED = 1, KVD_W_PACKED_GAMMA = 2 } kvd_weight_layout;

/* Operations whose workspace size kvd_workspace_bytes reports. */
typedef enum { KVD_OP_DECODE_ATTN = 0, KVD_OP_CACHED_ATTN = 1, KVD_OP_FUSED = 2 } kvd_op;

/* One attention layer's shape.
 *   d_model     residual width; a positive multiple of 64.
 *   n_q_heads   query heads; a positive multiple of n_kv_heads, with
 *               n_q_heads / n_kv_heads <= 16.
 *   n_kv_heads  key/value heads, >= 1.
 *   head_dim    64, 128 or 256.
 *   rms_eps     RMSNorm epsilon, finite and >= 0.
 *   rope_theta  RoPE base, finite and > 0.
 *   dtype       a kvd_dtype.
 *   w_layout    a kvd_weight_layout; the packed layouts require KVD_BF16.   */
typedef struct {
  int32_t d_model;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  float rms_eps;
  double rope_theta;
  int32_t dtype;
  int32_t w_layout;
} kvd_attn_shape;

/* A stored K/V block: k and v each [B][n_kv_heads][t_cap][head_dim] in the
 * shape dtype.  A call touches rows t_off .. t_off+T-1 of every (b, head),
 * which requires 0 <= t_off and t_off + T <= t_cap.                          */
typedef struct {
  void* k;
  void* v;
  int32_t t_cap;
  int32_t t_off;
} kvd_kv_view;

/* RECOMPUTE_KV (Algorithm 1; Eqs. k_recon, v_recon): for each sequence b < B
 * and residual row t < T,
 *   K[b][j][t_off+t] = RoPE(hbar W_k^(j), pos0[b]+t),  V[b][j][t_off+t] = hbar W_v^(j),
 * hbar = RMSNorm(h[b][t]).  This is also the prefill path (the K/V a cache
 * would have stored).  Every producer runs the same arithmetic (one MFMA chain
 * over d_model per output element, one sum-of-squares order), so prefill,
 * recompute, kvd_project_qkv's K/V and the fused kernel's K/V are bit-identical
 * for the same residual row and position (Prop. reconstruction).  A bf16 call of
 * few rows (at most 512 workgroups of 32 K/V rows x up to 16 tokens, 1024 for
 * head_dim 256: about 180 tokens of the Gemma-3-4B shape, 512 of the
 * Qwen2.5-1.5B shape) runs on the current-token projection's kernel, which
 * serves them at lower latency than the 64-token tile engine.
 *   h     [B][h_ld][d_model], h_ld >= T.      pos0  [B] int32.
 *   out   K/V view written at rows out->t_off .. out->t_off+T-1.
 * B == 0 or T == 0 is a no-op.                                                */
kvd_status kvd_recompute_kv(const kvd_attn_shape* shape, const void* h, int32_t h_ld,
                            const void* gamma, const void* w_k, const void* w_v,
                            const int32_t* pos0, int32_t B, int32_t T,
                            const kvd_kv_view* out, void* stream);

/* Current-token projections of a decode step (Algorithm 1; Eqs. q_proj,
 * k_proj, v_proj): for each sequence b,
 *   q_out[b][h] = RoPE(hbar W_q^(h), pos[b]),  hbar = RMSNorm(h_new[b]),
 * and, if kv_out is not NULL, the token's own K and V written at row
 * kv_out->t_off (exactly what kvd_recompute_kv gives for that row).
 *   h_new [B][d_model].   pos [B] int32.   q_out [B][n_q_heads][head_dim].   */
kvd_status kvd_project_qkv(const kvd_attn_shape* shape, const void* h_new, const void* gamma,
                           const void* w_q, const void* w_k, const void* w_v,
                           const int32_t* pos, int32_t B, void* q_out,
                           const kvd_kv_view* kv_out, void* stream);

/* The query projection alone (Sec. 3.1, Eq. q_proj; Algorithm 1's Q):
 *   q_out[b][h] = RoPE(hbar W_q^(h), pos[b]),  hbar = RMSNorm(h_new[b]).
 * The same call as kvd_project_qkv with kv_out == NULL (w_k / w_v unused), with
 * the argument list of the plain problem statement.
 *   h_new [B][d_model].   pos [B] int32.   q_out [B][n_q_heads][head_dim].   */
kvd_status kvd_project_q(const kvd_attn_shape* shape, const void* h_new, const void* gamma,
                         const void* w_q, const int32_t* pos, int32_t B, void* q_out, void* stream);

/* ATTENTION for one decode query per sequence and head (Eqs. attn_weights,
 * head_output) over T >= 1 stored keys: rows kv->t_off .. kv->t_off+T-1.
 * bf16: the keys of each (sequence, KV head) are cut into kvd_num_splits
 * contiguous ranges (about kvd_set_attn_workgroups workgroups over the call,
 * at most 32 ranges per (sequence, KV head)),
 * each streamed by one workgroup that keeps its next 16-key block's loads in
 * flight (HBM-bound: the read is Eq. read_bytes).  fp32: one split per
 * 64-key tile.
 * Split-K: partial softmax states go to the workspace; the workgroup that
 * writes the last partial of a (sequence, KV head) merges them into out in the
 * same kernel (an atomic split counter in the workspace; no spin-waits).
 * ws (256-byte aligned) must hold kvd_workspace_bytes(shape, KVD_OP_DECODE_ATTN,
 * B, T, 0) bytes.  Workspace contract: its first bytes hold split counters
 * ([B][n_kv_heads] uint64, padded to 256 bytes) that must be zero before the
 * first call that uses them (allocate the workspace zero-filled once); every
 * call leaves them zero.  The rest of the workspace is overwritten.  Their
 * place depends on B only, so attention calls of any key count and op (decode,
 * cached, fused) with the same B can share one workspace sized for the largest
 * of them, as a decode loop whose context grows does.  Calls sharing one
 * workspace must be ordered on one stream.  With out == NULL only
 * the partials are written (see kvd_combine) and the counters are not touched.
 *   q [B][n_q_heads][head_dim].   out [B][n_q_heads][head_dim].               */
kvd_status kvd_decode_attn(const kvd_attn_shape* shape, const void* q, const kvd_kv_view* kv,
                           int32_t B, int32_t T, void* out, void* ws, size_t ws_bytes,
                           void* stream);

/* The cached-K/V baseline: a standard KV-cache decode step's attention, which
 * reads every key and value from a persistent bf16 cache in HBM (the
 * B_read = 2 N n_kv d_head b bytes of Eq. read_bytes).  Same arguments and
 * kernels as kvd_decode_attn; shape->dtype must be KVD_BF16.  Workspace:
 * kvd_workspace_bytes(shape, KVD_OP_CACHED_ATTN, B, T, 0).                    */
kvd_status kvd_cached_attn(const kvd_attn_shape* shape, const void* q, const kvd_kv_view* kv,
                           int32_t B, int32_t T, void* out, void* ws, size_t ws_bytes,
                           void* stream);

/* One KV-Direct decode step's attention (Algorithm 1: RECOMPUTE_KV, CONCAT,
 * ATTENTION): keys and values are recomputed from the checkpointed residuals
 * h rows 0..T_rec-1 (positions pos0[b]+t) inside the kernel and attended from
 * LDS without being written to HBM, then concatenated with T_tail stored keys:
 * the tail view's rows t_off, t_off+1, ... taken modulo tail->t_cap, so a
 * bounded cache kept as a ring of t_cap slots is read oldest first from its
 * oldest slot t_off (0 <= t_off < t_cap, T_tail <= t_cap; a view with
 * t_off + T_tail <= t_cap is an ordinary contiguous block).  The tail is
 * typically the current token's own K/V from kvd_project_qkv (cache budget 0),
 * or Algorithm 1's bounded cache of recent tokens followed by the current one.
 *   T_rec >= 0, T_tail >= 0, T_rec + T_tail >= 1; tail may be NULL iff T_tail == 0.
 *   ws: kvd_workspace_bytes(shape, KVD_OP_FUSED, B, T_rec, T_tail) bytes.
 *   kv_debug: NULL in production.  If not NULL, the recomputed K/V are also
 *   written to it at rows kv_debug->t_off .. +T_rec-1 (for bit-identity checks).
 * Split-K as in kvd_decode_attn, one split per recomputed tile, on one of
 * four engines (see kvd_set_fused_tokens):
 *   - pair (bf16, head_dim 128, an even n_kv_heads, at most 6 query heads per
 *     KV head at common d_model): 128-token tiles of the K and V rows of two
 *     KV heads, when the call has at least 256 of them (B * n_kv_heads / 2 *
 *     ceil(T_rec / 128) >= 256); the same chunks and splits as wide;
 *   - wide (bf16, head_dim 128 / 256): 128-token tiles of K and V rows, when
 *     the call has at least 256 of them (B * n_kv_heads * ceil(T_rec / 128)
 *     >= 256: a full round of the chip);
 *   - split (bf16, head_dim 128 / 256, T_rec >= 1, T_tail <= 4, at most 256
 *     chunks per sequence) with 64-token chunks when 64-token tiles of both
 *     halves would fill at most 128 compute units (B * n_kv_heads *
 *     ceil(T_rec / 64) <= 128: sliding-window layers, short contexts), or when
 *     asked for (KVD_FUSED_SPLIT64; KVD_FUSED_SPLIT for 128-token chunks):
 *     each chunk runs as two workgroups, one recomputing its K rows
 *     and taking the scores and softmax, one recomputing its V rows and, once
 *     the first has published the probabilities through the workspace, the
 *     P V products.  The second waits for the first with a bounded wait
 *     (about 0.1 s); past it that split's partial is NaN, so out shows it;
 *   - 64-token tiles of K and V rows otherwise.
 * With bf16, T_rec >= 1 and T_tail <= 4 (a decode step's current token) the
 * tail joins the last tile's split on every engine: its rows are copied into
 * LDS while that tile is recomputed.  Otherwise the tail adds one split per
 * 64-row tile, each attended by a workgroup of its own (the hybrid cache
 * budget: recent tokens stored, older ones recomputed); with bf16 a remainder
 * of at most 4 rows joins the tile before it.  kvd_num_splits gives the count;
 * kvd_workspace_bytes covers every engine.
 * The workspace's split counters follow kvd_decode_attn's contract.
 * out == NULL writes only the split-K partials (see kvd_combine).
 * Supports both dtypes.                                                       */
kvd_status kvd_fused_recompute_attn(const kvd_attn_shape* shape, const void* q, const void* h,
                                    int32_t h_ld, const void* gamma, const void* w_k,
                                    const void* w_v, const int32_t* pos0, int32_t B,
                                    int32_t T_rec, const kvd_kv_view* tail, int32_t T_tail,
                                    void* out, void* ws, size_t ws_bytes,
                                    const kvd_kv_view* kv_debug, void* stream);

/* kvd_fused_recompute_attn without a workspace argument, for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  It allocates nothing.  Its split-K
 * partials and counters live in a static per-device scratch array of 32 MiB
 * (kvd_workspace_bytes(shape, KVD_OP_FUSED, B, T_rec, T_tail) must not exceed
 * 33554432, else KVD_ERR_WORKSPACE before any launch), held by every GPU the
 * library runs on until the process ends; its address is looked up once per
 * device on the first call.  Each call first clears its split counters with a
 * fill kernel, then runs exactly the kernels of kvd_fused_recompute_attn, so
 * out is bit-identical to that call's.  out must not be NULL (the splits are
 * always merged in the kernel); there is no kv_debug.  All calls on one GPU
 * share the one array: calls that overlap on a GPU (concurrent streams,
 * threads or processes' graph replays in flight together) race and give
 * wrong results; order them on one stream.  Other arguments as in
 * kvd_fused_recompute_attn.                                                   */
kvd_status kvd_fused_recompute_attn_noalloc(const kvd_attn_shape* shape, const void* q, const void* h,
                                            int32_t h_ld, const void* gamma, const void* w_k,
                                            const void* w_v, const int32_t* pos0, int32_t B,
                                            int32_t T_rec, const kvd_kv_view* tail, int32_t T_tail,
                                            void* out, void* stream);

/* A sliding-window layer's decode-step attention (Sec. 3.2, the sliding-window
 * boundary and Eq. sw_error; Sec. 5, the sliding-window limitation): of the
 * T = T_rec + T_tail keys that kvd_fused_recompute_attn would attend (residual
 * rows 0..T_rec-1 recomputed, then the stored tail rows), only the newest
 * min(T, window) take part (the local attention mask), and the key with index i
 * inside that window (i = 0 for the oldest kept key) is rotated by R_i, not by
 * its absolute position (window-relative RoPE).  The max(0, T - window) oldest
 * keys are dropped, recomputed rows first: the first kept residual row is
 * recomputed at position 0, the next at 1, and so on.  Stored tail rows that are
 * kept must carry the same window-relative rotation (e.g. the current token's K
 * from kvd_project_qkv at position min(T, window) - 1), and so must q.
 *   window >= 1.  Other arguments as in kvd_fused_recompute_attn (no pos0: the
 *   positions are window indices; no kv_debug).
 *   ws: kvd_workspace_bytes(shape, KVD_OP_FUSED, B, T_rec', T_tail') for the
 *   kept counts; the value for (T_rec, T_tail) always suffices.  Split counters
 *   as in kvd_decode_attn.                                                    */
kvd_status kvd_fused_window_attn(const kvd_attn_shape* shape, const void* q, const void* h,
                                 int32_t h_ld, const void* gamma, const void* w_k,
                                 const void* w_v, int32_t B, int32_t T_rec,
                                 const kvd_kv_view* tail, int32_t T_tail, int32_t window,
                                 void* out, void* ws, size_t ws_bytes, void* stream);

/* STORE_RESIDUAL (Algorithm 1; Eq. res_mem): checkpoint each sequence's
 * current residual, ckpt[b][row][:] = h_new[b][:] for b < B, in the shape
 * dtype.  A bounded cache (Algorithm 1 with budget > 0) stores every token's
 * residual when the token arrives, since its h^(l) exists only at that step,
 * and recomputes from it once the token is evicted from the cache.
 *   h_new [B][d_model].   ckpt [B][c_ld][d_model], 0 <= row < c_ld; must not
 *   overlap h_new.   B == 0 is a no-op.                                       */
kvd_status kvd_store_residual(const kvd_attn_shape* shape, const void* h_new, void* ckpt, int32_t c_ld,
                              int32_t row, int32_t B, void* stream);

/* Weight packing (done once per frozen weight matrix; the weights of the paper's
 * projections are fixed at inference, Sec. 3.2): rewrites a row-major
 * [rows][d_model] bf16 matrix into the order the MFMA kernels read it in, so
 * that every 64-lane load of a weight operand is one contiguous 1 KiB block:
 * block (r, c), r < rows/32, c < d_model/16, is 512 elements at offset
 * (r * d_model/16 + c) * 512, and its element 8*l + e (lane l < 64, e < 8) is
 * W[32 r + l % 32][16 c + 8 (l / 32) + e].  A head's rows start at the same
 * element offset (head * head_dim * d_model) as in the row-major matrix.
 * rows must be a positive multiple of 32; packed holds rows * d_model bf16 and
 * must not alias w.  shape->dtype must be KVD_BF16 (w_layout is ignored).    */
kvd_status kvd_pack_weights(const kvd_attn_shape* shape, const void* w, int32_t rows, void* packed,
                            void* stream);

/* kvd_pack_weights of W diag(gamma) for the KVD_W_PACKED_GAMMA layout: element
 * (f, k) of the packed matrix is bf16(W[f][k] * gamma[k]) (the product of the two
 * bf16 values is exact in fp32, then rounded to nearest even), in the block
 * order of kvd_pack_weights.  Pack W_q, W_k and W_v of a layer with that
 * layer's RMSNorm weight gamma ([d_model] bf16).  The RMSNorm of Eq. rmsnorm is
 * gamma * h / rms(h); moving gamma into the weights leaves each projection's
 * value unchanged up to rounding and lets the kernels use the residual rows as
 * MFMA operands as they are.  packed must alias neither w nor gamma.         */
kvd_status kvd_pack_weights_gamma(const kvd_attn_shape* shape, const void* w, const void* gamma, int32_t rows,
                                  void* packed, void* stream);

/* kvd_pack_weights for any bf16 matrix [rows][cols] (rows % 32 == 0,
 * cols % 16 == 0): block (r, c) of 32 rows x 16 columns is 512 elements at
 * offset (r * cols/16 + c) * 512 in MFMA A-operand lane order.  Used for the
 * block forward's W_o [d_model][n_q*head_dim] and W_down [d_model][d_ff], whose
 * rows are not d_model long.  packed must not alias w.                       */
kvd_status kvd_pack_matrix(const void* w, int32_t rows, int32_t cols, void* packed, void* stream);

/* The single-checkpoint scheme (Eq. res_mem: one residual vector per token
 * serves all layers; Algorithm 1 otherwise stores a residual per layer):
 * h^(l+1) of every position from h^(l), by one pre-norm transformer block
 * (Sec. 3.1, Eqs. q_proj, k_proj, v_proj, attn_weights, head_output,
 * attn_sublayer, mlp_sublayer).  Running it for layers 0 .. l-1 recomputes h^(l)
 * from the checkpoint h^(0).  For each sequence b and position t (at pos0[b]+t):
 *   hbar = RMSNorm(h; gamma_attn); q, K, V as kvd_recompute_kv / kvd_project_qkv
 *   compute them (the same tile engine and arithmetic); heads = causal attention
 *   (position t attends positions <= t); hhat = h + heads W_o^T;
 *   h_out = hhat + (SiLU(xbar W_gate^T) * (xbar W_up^T)) W_down^T,
 *   xbar = RMSNorm(hhat; gamma_mlp).
 * The MLP's form is not given by the paper; this is the SiLU-gated MLP of the
 * LLaMA and Qwen families it evaluates.  Weights are [out][in]: W_q
 * [n_q*hd][d], W_k/W_v [n_kv*hd][d], W_o [d][n_q*hd], W_gate/W_up [d_ff][d],
 * W_down [d][d_ff]; shape->w_layout applies to all of them (packed: each
 * through kvd_pack_weights / kvd_pack_matrix).  bf16 only; head_dim 128 or
 * 256; d_model % 512 == 0; d_ff % 256 == 0.  q, K, V, the heads, hhat and the
 * MLP activation are rounded to bf16 between kernels (RNE), accumulation fp32.
 *   h_in, h_out [B][T][d_model] (must not overlap).   pos0 [B] int32.
 *   ws: kvd_block_workspace_bytes(shape, d_ff, B, T) bytes, 256-byte aligned,
 *   overwritten.  B == 0 or T == 0 is a no-op.                                */
typedef struct {
  const void* gamma_attn;
  const void* w_q;
  const void* w_k;
  const void* w_v;
  const void* w_o;
  const void* gamma_mlp;
  const void* w_gate;
  const void* w_up;
  const void* w_down;
  int32_t d_ff;
} kvd_block_weights;

kvd_status kvd_block_forward(const kvd_attn_shape* shape, const kvd_block_weights* w,
                             const void* h_in, void* h_out, const int32_t* pos0, int32_t B,
                             int32_t T, void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes of kvd_block_forward (0 on invalid arguments).              */
size_t kvd_block_workspace_bytes(const kvd_attn_shape* shape, int32_t d_ff, int32_t B, int32_t T);

/* Merge step of split-K attention: out[b][h] = sum_s w_s acc_s / sum_s w_s l_s
 * with w_s = 2^(m_s - max_s m_s), over the S partial softmax states that a
 * preceding kvd_decode_attn / kvd_cached_attn / kvd_fused_recompute_attn call
 * (with out == NULL) left in ws, in a fixed order (deterministic; the same
 * arithmetic as the merge those calls run themselves when out != NULL).  S is
 * that call's kvd_num_splits.  Lets a caller time or schedule the merge
 * separately.                                                                 */
kvd_status kvd_combine(const kvd_attn_shape* shape, int32_t B, int32_t S, const void* ws,
                       size_t ws_bytes, void* out, void* stream);

/* Workspace bytes an attention call needs (0 on invalid arguments).  For
 * KVD_OP_DECODE_ATTN / KVD_OP_CACHED_ATTN, T_main is T and T_tail must be 0;
 * for KVD_OP_FUSED they are T_rec and T_tail.                                 */
size_t kvd_workspace_bytes(const kvd_attn_shape* shape, int32_t op, int32_t B, int32_t T_main,
                           int32_t T_tail);

/* Number of split-K partitions an attention call uses (0 on invalid arguments). */
int32_t kvd_num_splits(const kvd_attn_shape* shape, int32_t op, int32_t B, int32_t T_main,
                       int32_t T_tail);

/* Tuning of the bf16 stored-K/V attention (kvd_decode_attn, kvd_cached_attn):
 * the number of workgroups its split policy aims for over the whole call
 * (B * n_kv_heads * splits; default 256, one per MI355X compute unit;
 * target <= 0 restores the default).  Returns the previous value.  The setting
 * is process-wide and changes kvd_num_splits / kvd_workspace_bytes of those
 * ops: query workspace sizes after setting it, and do not change it while
 * calls that share a workspace are in flight.  Results are exact for every
 * setting (only the key ranges of the splits move).                          */
int32_t kvd_set_attn_workgroups(int32_t target);

/* Tuning of kvd_fused_recompute_attn and kvd_fused_window_attn: the recomputed
 * tokens per workgroup.  0 (the default) chooses per call, 128 asks for the
 * wide engine wherever it exists (bf16, head_dim 128 / 256, its LDS within
 * the limit; elsewhere 64 is used), KVD_FUSED_PAIR for the pair engine
 * wherever it exists (elsewhere the wide engine, else 64), KVD_FUSED_SPLIT /
 * KVD_FUSED_SPLIT64 for the split engine with 128- / 64-token chunks wherever
 * a call can run on it (elsewhere 64), 64 for the 64-token tiles;
 * other values mean 0.  Returns the previous setting.  Process-wide: it
 * changes kvd_num_splits of KVD_OP_FUSED (not kvd_workspace_bytes, which
 * covers every engine).  All engines give K/V bit-identical to
 * kvd_recompute_kv; the attention output differs by rounding only (other
 * split boundaries).                                                         */
#define KVD_FUSED_SPLIT (-128)
#define KVD_FUSED_SPLIT64 (-64)
#define KVD_FUSED_PAIR (-2)
int32_t kvd_set_fused_tokens(int32_t tokens);

const char* kvd_status_str(kvd_status status);
const char* kvd_last_error(void);
int kvd_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KVD_H */
