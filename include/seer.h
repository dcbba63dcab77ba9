/*
 * seer.h -- C ABI of the Seer hot path on MI355X (gfx950).
 *
 * Seer ("Seeing the End at Step Zero") shortens the fixed generation window
 * of a diffusion multimodal LLM: at denoising step 0 the MLP of an early layer
 * exposes, per window position, a near-zero activation count; an SNR
 * jump/plateau test on that count finds where the semantic text ends; the
 * suffix is cut once and every later layer and step runs on the shorter,
 * compacted batch (Sec. 3.2-3.5 of the paper).
 *
 * Entry points (all asynchronous on the given HIP stream):
 *   seer_prepack_weights       one-time weight layout for the layer kernels
 *   seer_layer_status_reset    clear the status word of a layer workspace
 *   seer_layer_forward_varlen  one bidirectional transformer layer over
 *                              packed variable-length sequences, with the
 *                              optional fused near-zero activation count
 *   seer_step0_detect          the SNR boundary criterion per sequence
 *   seer_layer_forward_detect  the detection layer: count, criterion, and a
 *                              down projection truncated to the kept rows
 *   seer_batch_repack          padding-waste-aware routing plus compaction
 *   seer_kv_export,            truncated steps on the window rows with the
 *   seer_layer_forward_cached  prefix keys/values cached (Appendix D)
 *   seer_graph_*               record a launch sequence once, replay it
 *                              (graph-compatible paths, Sec. 3.5)
 *   seer_lm_head_prepack,      synthetic LM head (one-time weight layout;
 *   seer_lm_head_predict,      argmax + confidence) and
 *   seer_remask_step           low-confidence remasking between steps
 *
 * Conventions shared by every call:
 *   - Buffers are owned by the caller.  Pointers are device pointers unless a
 *     parameter says "host".  The library never allocates or frees caller
 *     memory; layer scratch comes from a caller workspace sized by
 *     seer_layer_workspace_bytes().
 *   - Row-major everywhere, except the packed weights the prepack calls
 *     produce.  Weights are given in the [out, in] layout (input features
 *     contiguous).  Element type is given by seer_dims.dtype: bf16 (raw
 *     16-bit brain-float bits) or fp32.  Counts, offsets and lengths are int32.
 *   - Packed sequences: sequence b occupies rows [cu_seqlens[b], cu_seqlens[b+1])
 *     of a row buffer; cu_seqlens[0] == 0 and the array is non-decreasing.
 *     cu_seqlens lives in device memory and is read by the kernels, so the
 *     host never needs the real row count: it passes an upper bound that
 *     sizes the launch grids.
 *   - Return value: 0 on success, a negative SEER_E* code otherwise.  On error
 *     nothing is launched and seer_last_error() (per host thread) describes
 *     the problem.  Errors detected on the device (a buffer too small for the
 *     routed layout) are reported through seer_route_ctrl.status.
 *   - Outputs are valid once the stream reaches the point of the call.
 *     Calls on distinct streams with distinct workspaces may run concurrently.
 */
#ifndef SEER_H_
#define SEER_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define SEER_OK            0
#define SEER_EINVAL       -1   /* bad argument (null pointer, bad size, ...) */
#define SEER_EUNSUPPORTED -2   /* shape or dtype the library has no kernel for */
#define SEER_EWORKSPACE   -3   /* workspace or destination buffer too small */
#define SEER_EHIP         -4   /* a HIP runtime call failed */

/* ---- element types ----------------------------------------------------- */
#define SEER_DTYPE_BF16 1
#define SEER_DTYPE_F32  2

/* Layer geometry.  d_model = n_heads * head_dim.
 * bf16 kernels need d_model % 256 == 0, d_ff % 128 == 0, head_dim == 128.
 * fp32 kernels accept any d_model, d_ff and head_dim <= 128 (head_dim % 4 == 0). */
typedef struct seer_dims {
  int32_t d_model;
  int32_t n_heads;
  int32_t head_dim;
  int32_t d_ff;        /* SwiGLU intermediate size I */
  int32_t dtype;       /* SEER_DTYPE_* */
  float rms_eps;       /* RMSNorm epsilon (1e-5 for the LLaDA-shaped layer) */
  float rope_theta;    /* 0: no positional encoding (the paper's layer equations have
                          none).  > 1: rotary embedding of q and k (RoFormer's
                          definition, rotate-half pairs): features j and j + head_dim/2
                          of each head turn by pos * rope_theta^(-2 j / head_dim), pos
                          being the row's index in its sequence (plus the cached prefix
                          length in seer_layer_forward_cached).  The angle is reduced in
                          fp64 and evaluated by the hardware sine/cosine in fp32. */
} seer_dims;

/* Source weights of one layer (device pointers, dtype = dims.dtype, [out, in]):
 * wq, wk, wv, wo [d, d]; wg, wu [I, d]; wd [d, I].  g1, g2: fp32 RMSNorm gains
 * [d] before attention and before the MLP, or NULL for unit gains. */
typedef struct seer_layer_weights {
  const void* wq;
  const void* wk;
  const void* wv;
  const void* wo;
  const void* wg;
  const void* wu;
  const void* wd;
  const float* g1;
  const float* g2;
} seer_layer_weights;

/* Size in bytes of the prepacked weights of one layer. */
size_t seer_prepacked_bytes(const seer_dims* dims);

/* Repack one layer's weights into the kernels' layout in `dst` (device,
 * seer_prepacked_bytes() bytes, 256-byte aligned): q/k/v stacked, gate and up
 * rows interleaved in blocks of 32 so that one tile holds matching gate and
 * up columns, and the RMSNorm gains folded into the input columns of the
 * projections they feed (exact for unit gains).  bf16 layers also store every
 * matrix in the matrix cores' operand order (one 1 KiB block per 32 output
 * rows and 16 input columns) with the q and k rows of each head in 32-row
 * block order 0, 2, 1, 3; the layout is private to the library and may change
 * with the ABI version.  The source is not modified. */
int seer_prepack_weights(const seer_dims* dims, const seer_layer_weights* src,
                         void* dst, size_t dst_bytes, hipStream_t stream);

/* Workspace bytes needed by seer_layer_forward_varlen for up to max_rows
 * packed rows (qkv, attention output, post-attention residual, SwiGLU
 * activations and two per-row RMS statistics), plus a 256-byte header and,
 * for bf16 layers, 64 MiB for the fp32 partial sums of projections that split
 * their K dimension (those whose 256x256 output tiles would fill at most a
 * third of the GPU's compute units: few rows, as in prefix-cached steps).
 *
 * Status word: the int32 at byte 0 of the workspace (for every rows bound).
 * Layer calls only ever set bits in it (atomic OR), so it accumulates over
 * every call made on the workspace until seer_layer_status_reset() clears it;
 * a new allocation holds arbitrary bits until then.  Bits:
 *   SEER_STATUS_V_RANGE  a bf16 layer stored a value of V (the attention
 *                        values, kept in fp16 for the fp16 P V product) whose
 *                        magnitude exceeded 65504, fp16's largest finite
 *                        value: it was stored rounded (+-65504 or +-inf) and
 *                        the attention output of its sequence and head is not
 *                        meaningful.  Values below 2^-14 are kept as fp16
 *                        subnormals (absolute precision 2^-24), not flagged. */
#define SEER_STATUS_V_RANGE 1
size_t seer_layer_workspace_bytes(const seer_dims* dims, int32_t max_rows);

/* Clear the status word of a layer workspace (device, 256-byte aligned, at
 * least 256 bytes), asynchronously on `stream` (a kernel, so it can be
 * recorded).  Errors: EINVAL (NULL or misaligned), EWORKSPACE (too small). */
int seer_layer_status_reset(void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Byte offsets of the intermediates that the last seer_layer_forward_varlen
 * call on a workspace left there, for a call made with total_rows_ub ==
 * max_rows (the layout depends on that bound; bytes [0, 256) are the header
 * with the status word).  Element type dims.dtype unless noted:
 *   offsets[0] qkv  [max_rows, 3*d_model]   q | k | v after the folded RMSNorm
 *                                           (bf16 layers: v is stored as fp16,
 *                                           the type of the attention's P V product)
 *   offsets[1] o    [max_rows, d_model]     attention output (pre projection)
 *   offsets[2] h1   [max_rows, d_model]     x + o Wo^T
 *   offsets[3] act  [max_rows, d_ff]        silu(gate) * up
 *   offsets[4] fp32 [max_rows]              1/rms of x
 *   offsets[5] fp32 [max_rows]              1/rms of h1 (as the MLP reads it)
 *   offsets[6] bf16 [max_rows, d_model]     low part of h1, bf16(h1 - bf16(h1)):
 *                                           the final residual add uses
 *                                           offsets[2] + offsets[6], h1 to
 *                                           ~2^-17 (bf16 layers; fp32 layers:
 *                                           equal to offsets[2])
 *   offsets[7] total workspace bytes
 * Rows [0, cu_seqlens[batch]) of the last call are valid.  Meant for
 * inspection and teacher-forced checks.  Errors: EINVAL, EUNSUPPORTED. */
int seer_layer_workspace_offsets(const seer_dims* dims, int32_t max_rows, size_t offsets[8]);

/* One bidirectional transformer layer over packed sequences: the work every
 * denoising step repeats for every position of the window (Sec. 3.1):
 *     a   = RMSNorm(x) * g1;   q,k,v = a Wq^T, a Wk^T, a Wv^T
 *     o   = per head softmax(q k^T / sqrt(head_dim)) v, over all keys of the
 *           same sequence (no causal mask, Sec. 3.6 attention equations)
 *     h1  = x + o Wo^T
 *     b   = RMSNorm(h1) * g2;  act = silu(b Wg^T) * (b Wu^T)
 *     y   = h1 + act Wd^T
 * Precision (bf16 layers): operands bf16, accumulation fp32; q, k, o, h1
 * and act are rounded to bf16 where they feed a matrix product; v and the
 * probabilities of the attention-weighted sum are kept in fp16 (so |v| must
 * stay within fp16's range: a larger value sets SEER_STATUS_V_RANGE in the
 * workspace status word); the residual h1 enters the final add as a bf16
 * high/low pair (exact to ~2^-17).
 * x_in, x_out: [total_rows_ub, d_model] rows (may not alias).  Only rows
 * [0, cu_seqlens[batch]) are read and written.
 * seqused: optional [batch]; when given, rows at index >= seqused[b] inside
 * sequence b are padding: they are masked as keys (the attention-mask rewrite
 * of the static-bucket path, Sec. 3.5) and receive no attention output.
 * act_count: optional [total_rows_ub] int32; when non-NULL the call zeroes it
 * and stores, per row, the number of SwiGLU activations with
 * |act| < act_eps (strict), counted on the fp32 values before rounding --
 * the per-position MLP sparsity statistic of Sec. 3.2-3.3.
 * workspace: >= seer_layer_workspace_bytes(dims, total_rows_ub) bytes,
 * 256-byte aligned.  Errors: EINVAL (null pointers, batch < 1,
 * total_rows_ub < 1), EUNSUPPORTED (dims; bf16 with total_rows_ub x
 * max(3 d_model, d_ff) x 2 bytes >= 4 GiB: the kernels use 32-bit row
 * offsets), EWORKSPACE. */
int seer_layer_forward_varlen(const seer_dims* dims, const void* w_packed,
                              const void* x_in, void* x_out, int32_t total_rows_ub,
                              const int32_t* cu_seqlens, const int32_t* seqused,
                              int32_t batch, float act_eps, int32_t* act_count,
                              void* workspace, size_t workspace_bytes,
                              hipStream_t stream);

/* seer_layer_forward_varlen for callers that cannot allocate (code recorded
 * into a graph, tight serving loops, hosts that forbid allocation): the same
 * kernels, with the workspace taken from a device array inside the library
 * instead of a caller buffer.  The array holds 256 MiB (268435456 bytes) per
 * GPU the library runs on, from its first call on that device until the
 * process ends; the call allocates nothing (the array's device address is
 * looked up once per device, on the first call made with it current).
 * Arguments as in seer_layer_forward_varlen, without the workspace; status:
 * optional device int32 that receives the SEER_STATUS_* bits of this call
 * (atomic OR; the caller zeroes it), NULL for none.  Limit: a rows bound
 * whose seer_layer_workspace_bytes(dims, total_rows_ub) exceeds 268435456 is
 * refused with SEER_EWORKSPACE (the LLaDA-8B layer shape, d_model 4096 and
 * d_ff 12288 in bf16, takes up to 2730 rows).  Every call on one GPU shares
 * that GPU's array: calls that overlap in time on one GPU (other streams,
 * other host threads) race and must not be issued.  Intermediates are not
 * exposed (seer_layer_workspace_offsets does not apply).  Errors: as
 * seer_layer_forward_varlen; EWORKSPACE (rows bound too large), EHIP (the
 * array could not be located on the current device). */
int seer_layer_forward_varlen_noalloc(const seer_dims* dims, const void* w_packed, const void* x_in,
                                      void* x_out, int32_t total_rows_ub, const int32_t* cu_seqlens,
                                      const int32_t* seqused, int32_t batch, float act_eps,
                                      int32_t* act_count, int32_t* status, hipStream_t stream);

/* As seer_layer_forward_varlen, recording events[k] (created by the caller)
 * on `stream` around its kernels for live per-kernel timing:
 *   events[0] -> [1] RMS statistics of x       [1] -> [2] QKV GEMM
 *   events[2] -> [3] attention                 [3] -> [4] O GEMM + residual
 *   events[4] -> [5] RMS statistics of h1 (+ zeroing act_count)
 *   events[5] -> [6] gate/up GEMM + SwiGLU (+ count)
 *   events[6] -> [7] down GEMM + residual
 * A NULL entry is skipped (that point is not recorded): each record delays
 * the next launch by a few microseconds, so a caller timing one kernel
 * passes only the two events around it.
 * Errors: as seer_layer_forward_varlen, EINVAL if events is NULL. */
int seer_layer_forward_varlen_timed(const seer_dims* dims, const void* w_packed,
                                    const void* x_in, void* x_out, int32_t total_rows_ub,
                                    const int32_t* cu_seqlens, const int32_t* seqused,
                                    int32_t batch, float act_eps, int32_t* act_count,
                                    void* workspace, size_t workspace_bytes,
                                    hipStream_t stream, hipEvent_t events[8]);

/* Truncated step with the prefix's keys and values cached (the KV-cache
 * combination of Appendix D, compatibility with KV caching): the layer of
 * seer_layer_forward_varlen on rows that hold only the kept generation
 * window of each sequence, every row attending to the cached keys of its
 * sequence's prefix followed by the sequence's own keys.
 * x_in, x_out, total_rows_ub, cu_seqlens, seqused, batch, workspace: as in
 * seer_layer_forward_varlen, for the window rows (seqused[b] = real window
 * rows; padding rows are no keys and receive no attention output).
 * kv_cache: [kv_rows, 2 d_model] rows of K | V as seer_kv_export writes
 * them (bf16 layers: K bf16, V fp16; fp32 layers: fp32), 16-byte aligned;
 * sequence b's prefix is rows [cu_kv[b], cu_kv[b+1]) (cu_kv: [batch+1],
 * device, non-decreasing); kv_rows_ub >= cu_kv[batch] bounds it.
 * Given the cache of a full step over the same inputs, the outputs equal
 * that step's window rows.  No near-zero count (only step 0 counts).
 * Errors: as seer_layer_forward_varlen; EINVAL (kv_cache or cu_kv NULL,
 * kv_rows_ub < 0, misaligned cache), EUNSUPPORTED (kv_rows_ub * 2 d_model
 * >= 2^32). */
int seer_layer_forward_cached(const seer_dims* dims, const void* w_packed,
                              const void* x_in, void* x_out, int32_t total_rows_ub,
                              const int32_t* cu_seqlens, const int32_t* seqused,
                              int32_t batch, const void* kv_cache, const int32_t* cu_kv,
                              int32_t kv_rows_ub, void* workspace, size_t workspace_bytes,
                              hipStream_t stream);

/* Cache the prefix keys and values of the last layer call made on
 * `workspace` (with the same total_rows_ub): for sequence b, the K | V
 * columns of its first cu_kv[b+1] - cu_kv[b] rows (rows [cu_seqlens[b], ...)
 * of that call) go to kv_dst rows [cu_kv[b], cu_kv[b+1]) ([kv_rows, 2 d_model],
 * element types as in the call's qkv region).  kv_rows_ub >= cu_kv[batch]
 * sizes the launch.  Cache rows of a prefix longer than its sequence are left
 * untouched.  Errors: EINVAL (null pointers, batch < 1, total_rows_ub < 1,
 * kv_rows_ub < 0, misaligned workspace or kv_dst), EUNSUPPORTED (dims),
 * EWORKSPACE. */
int seer_kv_export(const seer_dims* dims, const void* workspace, size_t workspace_bytes,
                   int32_t total_rows_ub, const int32_t* cu_seqlens, int32_t batch,
                   const int32_t* cu_kv, int32_t kv_rows_ub, void* kv_dst,
                   hipStream_t stream);

/* SNR criterion parameters as exact rationals: tau_jump = tau_num/tau_den,
 * gamma = gamma_num/gamma_den; lookahead = size of the window W_i.
 * The paper's defaults are {3, 100, 3, 5, 3}. */
typedef struct seer_snr_params {
  int32_t tau_num;
  int32_t tau_den;
  int32_t gamma_num;
  int32_t gamma_den;
  int32_t lookahead;
} seer_snr_params;

/* SNR-aware boundary detection (Sec. 3.3).  For sequence b the window counts
 * are c_i = act_count[cu_seqlens[b] + win_off[b] + i], i in [0, win_len[b]),
 * and s_i = c_i / d_ff.  The boundary is the first i in [1, win_len-lookahead]
 * with  min(W_i) - s_{i-1} >= tau  and  max(W_i) - min(W_i) <= gamma * jump,
 * evaluated exactly in 64-bit integers (tau_den*jump >= tau_num*d_ff and
 * gamma_den*noise <= gamma_num*jump on the counts).  Outputs per sequence:
 * boundary[b] = i* (win_len[b] when no position qualifies) and
 * keep_len[b] = min(i* + 1, win_len[b]) (one extra token is kept).
 * Errors: EINVAL (null pointers, batch < 1, d_ff < 1, denominators < 1,
 * lookahead < 1, negative numerators). */
int seer_step0_detect(const int32_t* act_count, const int32_t* cu_seqlens,
                      const int32_t* win_off, const int32_t* win_len, int32_t batch,
                      int32_t d_ff, const seer_snr_params* params,
                      int32_t* boundary, int32_t* keep_len, hipStream_t stream);

/* The detection layer of step 0 (Sec. 3.2-3.5): seer_layer_forward_varlen
 * with the near-zero count (act_count required, seqused none), the SNR scan
 * of seer_step0_detect on those counts once the gate/up projection has
 * written them, and then the down projection + residual only where its rows
 * are kept.  The boundary is known before the layer's last GEMM, and the rows
 * past it are dropped by the compaction that follows, so that GEMM is
 * truncated already: with bf16 it computes the 256-row tiles of x_out that
 * hold a kept row, rows [cu_seqlens[b], cu_seqlens[b] + win_off[b] +
 * keep_len[b]) of sequence b, and leaves the rows of the other tiles
 * unwritten; fp32 computes every row.
 * Arguments: those of seer_layer_forward_varlen (seqused absent) and of
 * seer_step0_detect (d_ff = dims->d_ff).  Outputs: act_count, boundary and
 * keep_len; x_out on every kept row.  These equal, bit for bit, what
 * seer_layer_forward_varlen followed by seer_step0_detect gives with the same
 * total_rows_ub; x_out rows past a sequence's kept rows are unspecified.
 * The workspace holds the list of kept tiles (seer_layer_workspace_bytes
 * counts it).  Errors: those of the two calls. */
int seer_layer_forward_detect(const seer_dims* dims, const void* w_packed, const void* x_in,
                              void* x_out, int32_t total_rows_ub, const int32_t* cu_seqlens,
                              int32_t batch, float act_eps, int32_t* act_count,
                              const int32_t* win_off, const int32_t* win_len,
                              const seer_snr_params* params, int32_t* boundary,
                              int32_t* keep_len, void* workspace, size_t workspace_bytes,
                              hipStream_t stream);

/* As seer_layer_forward_detect, recording events[k] (created by the caller)
 * on `stream` for live per-kernel timing: events[0] .. [6] as in
 * seer_layer_forward_varlen_timed, then
 *   events[6] -> [7] SNR scan + list of kept row tiles
 *   events[7] -> [8] down GEMM + residual (kept tiles)
 * NULL entries are skipped, as there.
 * Errors: as seer_layer_forward_detect, EINVAL if events is NULL. */
int seer_layer_forward_detect_timed(const seer_dims* dims, const void* w_packed, const void* x_in,
                                    void* x_out, int32_t total_rows_ub, const int32_t* cu_seqlens,
                                    int32_t batch, float act_eps, int32_t* act_count,
                                    const int32_t* win_off, const int32_t* win_len,
                                    const seer_snr_params* params, int32_t* boundary,
                                    int32_t* keep_len, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream, hipEvent_t events[9]);

/* Routing policies (Sec. 3.4 and the system study of Sec. 4):
 * HYBRID = three-tier Static / Varlen / Eager routing by padding waste ratio;
 * NAIVE_PAD = every sequence padded to the bucket of the batch-max length;
 * VARLEN_ONLY = every sequence packed without padding. */
#define SEER_ROUTE_HYBRID      0
#define SEER_ROUTE_NAIVE_PAD   1
#define SEER_ROUTE_VARLEN_ONLY 2

/* Paths written to route[b*3+0]. */
#define SEER_PATH_STATIC 0
#define SEER_PATH_VARLEN 1
#define SEER_PATH_EAGER  2

typedef struct seer_repack_desc {
  int32_t policy;            /* SEER_ROUTE_* */
  int32_t tau_pad_num;       /* static path iff rho <= tau_pad_num/tau_pad_den */
  int32_t tau_pad_den;       /*   (paper default 1/5) */
  int32_t granule;           /* packed capacity rounded up to a multiple (>= 1) */
  int32_t row_bytes;         /* bytes per row, a positive multiple of 16 */
  int32_t dst_capacity_rows; /* rows available in every dst buffer */
  int32_t max_batch_hint;    /* unused, 0 */
  int32_t flags;             /* SEER_REPACK_* bits, 0 for the default layout */
} seer_repack_desc;

/* seer_repack_desc.flags: copy only the kept window rows of each sequence
 * (no prefix rows), the input layout of seer_layer_forward_cached. */
#define SEER_REPACK_WINDOW_ONLY 1

/* Control word written by seer_batch_repack: the routed shape of the batch,
 * so a host can pick the launch configuration of the next steps without
 * waiting for the data tensors (Sec. 3.5).  `ready` is written last. */
typedef struct seer_route_ctrl {
  int32_t total_rows;        /* cu_dst[batch] */
  int32_t capacity_rows;     /* total_rows rounded up to the granule */
  int32_t n_static;
  int32_t n_varlen;
  int32_t n_eager;
  int32_t n_groups;
  int32_t max_alloc;         /* largest per-sequence window allocation */
  int32_t status;            /* 0 ok, SEER_EWORKSPACE if dst was too small */
  int32_t ready;             /* 1 once the fields above are final */
  int32_t reserved[7];
} seer_route_ctrl;

/* Routing + in-GPU compaction (Sec. 3.4-3.5), one launch, no host sync.
 * Route: bucket(L) = smallest of {8,16,32,...} u {N_max} that is >= L
 * (N_max = max_b win_len[b]); sequences fall in coarse classes
 * k = ceil(log4 max(L,8)), one group per class; a group G with bucket B_G has
 * padding waste rho = 1 - sum L / (|G| B_G); path = eager if |G| == 1 or
 * max L <= 4, else static if rho <= tau_pad, else varlen.  route[b*3+0] =
 * path, route[b*3+1] = group id (ascending class order), route[b*3+2] =
 * rows allocated to the window (B_G on the static path, keep_len otherwise).
 * Compaction, for each of the n_buffers (src[i] -> dst[i]) pairs (host
 * arrays of device pointers, rows of desc->row_bytes bytes, src laid out by
 * cu_src): sequence b's first win_off[b] + keep_len[b] rows are copied to
 * rows [cu_dst[b], ...) and the rest of its allocation is zero-filled;
 * cu_dst[b+1] = cu_dst[b] + win_off[b] + alloc_b; seqused[b] =
 * win_off[b] + keep_len[b]; rows [cu_dst[batch], capacity) are zero-filled.
 * With SEER_REPACK_WINDOW_ONLY in desc->flags the prefix rows are left out:
 * rows [win_off[b], win_off[b] + keep_len[b]) of sequence b are copied,
 * cu_dst[b+1] = cu_dst[b] + alloc_b and seqused[b] = keep_len[b].
 * Order of sequences is preserved.  ctrl_dev (device) and ctrl_host
 * (host-pinned, hipHostMalloc'ed) are optional.  If the routed capacity
 * exceeds desc->dst_capacity_rows, nothing is copied, cu_dst is all zero and
 * ctrl.status = SEER_EWORKSPACE.  Errors: EINVAL (null pointers, batch < 1,
 * n_buffers < 1, bad desc fields). */
int seer_batch_repack(const seer_repack_desc* desc, const void* const* src,
                      void* const* dst, int32_t n_buffers, const int32_t* cu_src,
                      const int32_t* win_off, const int32_t* win_len,
                      const int32_t* keep_len, int32_t batch, int32_t* cu_dst,
                      int32_t* seqused, int32_t* route, seer_route_ctrl* ctrl_dev,
                      seer_route_ctrl* ctrl_host, hipStream_t stream);

/* ---- synthetic LM head and remasking sampler -----------------------------
 * Makes synthetic denoising steps differ (Sec. 3.1: every step predicts all
 * masked positions at once).  The paper leaves the sampler to its backbones;
 * this follows the low-confidence remasking of the LLaDA family with a random
 * head.  bf16 layers only.
 *
 * seer_lm_head_prepack: copy the head weight w_lm [vocab, d] (device, bf16,
 * row-major [out, in]) into `dst` (device, at least vocab * d * 2 bytes,
 * 256-byte aligned) in the matrix cores' operand order, the form
 * seer_lm_head_predict reads (same layout as the packed layer weights: one
 * 1 KiB block per 32 vocabulary rows and 16 input columns).  Once per head.
 * Errors: EINVAL (null pointers, alignment, dst_bytes too small),
 * EUNSUPPORTED (fp32, vocab, 4 GiB or more).
 *
 * seer_lm_head_predict: for rows r < cu_seqlens[batch] of x [rows_ub, d]:
 * logits l = RMSNorm(x_r) (unit gain, dims->rms_eps) . w_lm^T, w_lm [vocab, d]
 * bf16 ([out, in]) as packed by seer_lm_head_prepack (w_packed);
 * pred[r] = argmax_v l_v (the smallest v among equal
 * maxima), conf[r] = its softmax probability 1 / sum_v exp(l_v - l_max).
 * Logits are fp32 (bf16 products, fp32 accumulation) and never stored: the
 * GEMM epilogue keeps a {max, sum exp, argmax} partial per row and 64
 * columns, merged by a second kernel.  vocab % 256 == 0.  Workspace: at
 * least seer_lm_head_workspace_bytes(dims, vocab, rows_ub), 256-byte aligned.
 * Errors: EINVAL (null pointers, sizes < 1, alignment), EUNSUPPORTED (fp32,
 * vocab, w_packed or x of 4 GiB or more), EWORKSPACE.
 *
 * seer_remask_step: per sequence b (rows [cu_seqlens[b], cu_seqlens[b+1]), the
 * first min(seqused[b], max_used) of them real; seqused may be NULL): among
 * the real positions with tokens[r] == -1 (masked), n of them, commit the
 * k = ceil(n / steps_left) with the largest conf (ties to the smaller
 * position): tokens[r] = pred[r] (clamped to [0, vocab)).  Then write every
 * row of the sequence to x_next: emb[tokens[r]] if committed, the x0 row if
 * still masked, zero past the real rows.  x_next may alias x0 (a committed
 * row's x0 row is never read again).  max_used <= 8192.  Errors: EINVAL,
 * EUNSUPPORTED (fp32, max_used). */
size_t seer_lm_head_workspace_bytes(const seer_dims* dims, int32_t vocab, int32_t rows_ub);
int seer_lm_head_prepack(const seer_dims* dims, const void* w_lm, int32_t vocab, void* dst, size_t dst_bytes,
                         hipStream_t stream);
int seer_lm_head_predict(const seer_dims* dims, const void* w_packed, int32_t vocab, const void* x, int32_t rows_ub,
                         const int32_t* cu_seqlens, int32_t batch, int32_t* pred, float* conf, void* workspace,
                         size_t workspace_bytes, hipStream_t stream);
int seer_remask_step(const seer_dims* dims, const int32_t* cu_seqlens, const int32_t* seqused, int32_t batch,
                     int32_t max_used, int32_t steps_left, const int32_t* pred, const float* conf, int32_t* tokens,
                     const void* x0, const void* emb, int32_t vocab, void* x_next, hipStream_t stream);

/* ---- recorded launch sequences (Sec. 3.5) -------------------------------
 * The graph-compatible execution paths replay a fixed launch sequence.  Every
 * kernel here reads its row counts and sequence offsets from device memory
 * and sizes its grid from the rows_ub the host passes, so one recorded
 * sequence serves every batch whose routed capacity (seer_route_ctrl.
 * capacity_rows) is at most the rows_ub it was recorded with: a 1-D graph
 * shape per capacity.
 *
 * seer_graph_begin starts recording the calls issued on `stream` by the
 * calling host thread (HIP stream capture, thread-local mode); they are not
 * run.  Only asynchronous seer_* entry points (not the _timed variant) may be
 * issued on the stream until seer_graph_end, which closes the recording and
 * instantiates it.  seer_graph_launch runs one replay on `stream`; a replay
 * reads the current contents of every buffer that the recorded calls named,
 * so inputs are updated in place between replays.  The buffers must stay
 * allocated while the graph exists.  seer_graph_destroy frees the graph
 * (NULL: no-op).  Replays on one stream run in order; a graph must not be
 * replayed on two streams at once.
 * Errors: EINVAL (null stream for begin, stream already recording, null
 * graph), EHIP (the runtime refused the recording, e.g. a recorded call
 * failed or an unsupported API was used while recording).  After a failed
 * recorded call, seer_graph_end still ends the recording and returns EHIP. */
typedef struct seer_graph_* seer_graph_t;
int seer_graph_begin(hipStream_t stream);
int seer_graph_end(hipStream_t stream, seer_graph_t* graph);
int seer_graph_launch(seer_graph_t graph, hipStream_t stream);
int seer_graph_destroy(seer_graph_t graph);

/* Description of the last error on the calling host thread ("" if none). */
const char* seer_last_error(void);

/* ABI version of this library (major * 100 + minor). */
int32_t seer_abi_version(void);   /* 104: the detection layer (seer_layer_forward_detect) */

#ifdef __cplusplus
}
#endif

#endif /* SEER_H_ */
