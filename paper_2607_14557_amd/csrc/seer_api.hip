// C ABI of the Seer hot path: argument checks, workspace layout and the launch
// sequence of each entry point.  Kernels live in gemm_bf16.hip, attn_bf16.hip,
// f32_kernels.hip and rows.hip.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <string>

#include "../../include/seer.h"
#include "kernels.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return SEER_OK;
}

int hip_fail(const char* what) {
  const hipError_t e = hipGetLastError();
  return fail(SEER_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t up256(size_t n) { return (n + 255) / 256 * 256; }

int check_dims(const seer_dims* d) {
  if (!d) return fail(SEER_EINVAL, "dims is NULL");
  if (d->d_model <= 0 || d->n_heads <= 0 || d->head_dim <= 0 || d->d_ff <= 0)
    return fail(SEER_EINVAL, "dims must be positive (d_model=%d n_heads=%d head_dim=%d d_ff=%d)",
                d->d_model, d->n_heads, d->head_dim, d->d_ff);
  if (d->n_heads * d->head_dim != d->d_model)
    return fail(SEER_EINVAL, "n_heads * head_dim (%d) != d_model (%d)", d->n_heads * d->head_dim,
                d->d_model);
  if (!(d->rms_eps >= 0.0f) || !isfinite(d->rms_eps)) return fail(SEER_EINVAL, "rms_eps must be finite and >= 0");
  if (!(d->rope_theta >= 0.0f) || !isfinite(d->rope_theta) || (d->rope_theta > 0.0f && d->rope_theta <= 1.0f))
    return fail(SEER_EINVAL, "rope_theta must be 0 (no rotary embedding) or finite and > 1");
  if (d->rope_theta > 0.0f && d->head_dim % 2 != 0)
    return fail(SEER_EUNSUPPORTED, "the rotary embedding needs an even head_dim");
  if (d->dtype == SEER_DTYPE_BF16) {
    if (d->d_model % 256 != 0 || d->d_ff % 128 != 0 || d->head_dim != 128)
      return fail(SEER_EUNSUPPORTED,
                  "bf16 kernels need d_model %% 256 == 0, d_ff %% 128 == 0, head_dim == 128 "
                  "(got %d, %d, %d)", d->d_model, d->d_ff, d->head_dim);
  } else if (d->dtype == SEER_DTYPE_F32) {
    if (d->head_dim > 128) return fail(SEER_EUNSUPPORTED, "fp32 attention needs head_dim <= 128");
  } else {
    return fail(SEER_EUNSUPPORTED, "unknown dtype %d", d->dtype);
  }
  return SEER_OK;
}

struct WsLayout {
  size_t qkv, o, h1, act, inv1, inv2, h1lo, pos, freq, tmap, part, part_bytes, total;
};

// bf16 layers: fp32 partial tiles of the GEMMs that split K (launches whose
// tiles fill at most half of the CUs; at most one 256x256 fp32 tile per
// workgroup of one round, 256 CUs x 256 KiB).
constexpr size_t PART_BYTES = (size_t)64 << 20;

// The first 256 bytes of a layer workspace are a header whose first int32 is
// the status word (same place for every rows bound, so it persists across
// calls of different sizes on one workspace).
constexpr size_t WS_HEADER = 256;

WsLayout ws_layout(const seer_dims* d, int rows) {
  const size_t es = d->dtype == SEER_DTYPE_BF16 ? 2 : 4;
  const size_t R = (size_t)(rows > 0 ? rows : 0);
  WsLayout L;
  size_t off = WS_HEADER;
  L.qkv = off; off = up256(off + R * 3 * d->d_model * es);
  L.o = off;   off = up256(off + R * d->d_model * es);
  L.h1 = off;  off = up256(off + R * d->d_model * es);
  L.act = off; off = up256(off + R * d->d_ff * es);
  L.inv1 = off; off = up256(off + R * 4);
  L.inv2 = off; off = up256(off + R * 4);
  // bf16 layers keep the low part of h1, bf16(h1 - bf16(h1)), for the final
  // residual add
  L.h1lo = d->dtype == SEER_DTYPE_BF16 ? off : L.h1;
  if (d->dtype == SEER_DTYPE_BF16) off = up256(off + R * d->d_model * 2);
  // rotary embedding: per-row positions and the per-pair frequencies
  L.pos = off;  off = up256(off + R * 4);
  L.freq = off; off = up256(off + 64 * 8);
  // the detection layer's list of kept 256-row tiles
  L.tmap = off; off = up256(off + (1 + (R + 255) / 256) * 4);
  L.part = off;
  L.part_bytes = d->dtype == SEER_DTYPE_BF16 ? PART_BYTES : 0;
  off = up256(off + L.part_bytes);
  L.total = off;
  return L;
}

}  // namespace

extern "C" {

const char* seer_last_error(void) { return g_err.c_str(); }

int32_t seer_abi_version(void) { return 104; }

size_t seer_prepacked_bytes(const seer_dims* dims) {
  if (check_dims(dims) != SEER_OK) return 0;
  return seer::packed_layout(dims->d_model, dims->d_ff, dims->dtype == SEER_DTYPE_BF16).total_bytes;
}

int seer_prepack_weights(const seer_dims* dims, const seer_layer_weights* src, void* dst,
                         size_t dst_bytes, hipStream_t stream) {
  int rc = check_dims(dims);
  if (rc) return rc;
  if (!src || !dst) return fail(SEER_EINVAL, "src/dst is NULL");
  if (!src->wq || !src->wk || !src->wv || !src->wo || !src->wg || !src->wu || !src->wd)
    return fail(SEER_EINVAL, "a weight pointer is NULL");
  if (!aligned(dst, 256)) return fail(SEER_EINVAL, "dst must be 256-byte aligned");
  const bool bf16 = dims->dtype == SEER_DTYPE_BF16;
  const size_t need = seer::packed_layout(dims->d_model, dims->d_ff, bf16).total_bytes;
  if (dst_bytes < need) return fail(SEER_EWORKSPACE, "dst holds %zu bytes, need %zu", dst_bytes, need);
  seer::PrepackParams p{};
  p.wq = src->wq; p.wk = src->wk; p.wv = src->wv; p.wo = src->wo;
  p.wg = src->wg; p.wu = src->wu; p.wd = src->wd;
  p.g1 = src->g1; p.g2 = src->g2;
  p.dst = dst;
  p.d = dims->d_model;
  p.d_ff = dims->d_ff;
  p.bf16 = bf16;
  if (seer::launch_prepack(p, stream)) return hip_fail("prepack launch");
  return ok();
}

size_t seer_layer_workspace_bytes(const seer_dims* dims, int32_t max_rows) {
  if (check_dims(dims) != SEER_OK || max_rows < 0) return 0;
  return ws_layout(dims, max_rows).total;
}

int seer_layer_status_reset(void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!workspace) return fail(SEER_EINVAL, "workspace is NULL");
  if (!aligned(workspace, 256)) return fail(SEER_EINVAL, "workspace must be 256-byte aligned");
  if (workspace_bytes < WS_HEADER)
    return fail(SEER_EWORKSPACE, "workspace holds %zu bytes, need at least %zu", workspace_bytes, WS_HEADER);
  // a kernel, not a memset, so that the call can be recorded
  if (seer::launch_zero_i32(static_cast<int32_t*>(workspace), 1, stream)) return hip_fail("zero launch");
  return ok();
}

int seer_layer_workspace_offsets(const seer_dims* dims, int32_t max_rows, size_t offsets[8]) {
  int rc = check_dims(dims);
  if (rc) return rc;
  if (!offsets || max_rows < 0) return fail(SEER_EINVAL, "offsets is NULL or max_rows < 0");
  const WsLayout L = ws_layout(dims, max_rows);
  offsets[0] = L.qkv; offsets[1] = L.o; offsets[2] = L.h1;
  offsets[3] = L.act; offsets[4] = L.inv1; offsets[5] = L.inv2;
  offsets[6] = L.h1lo; offsets[7] = L.total;
  return ok();
}

static int check_snr(const seer_snr_params* params) {
  if (params->tau_den < 1 || params->gamma_den < 1 || params->tau_num < 0 || params->gamma_num < 0)
    return fail(SEER_EINVAL, "tau/gamma must be non-negative rationals with positive denominators");
  if (params->lookahead < 1) return fail(SEER_EINVAL, "lookahead must be >= 1");
  return SEER_OK;
}

// The SNR scan run inside the detection layer, between the count and the
// down projection.
struct DetectStep {
  const int32_t* win_off;
  const int32_t* win_len;
  const seer_snr_params* snr;
  int32_t* boundary;
  int32_t* keep_len;
};

static int layer_forward_impl(const seer_dims* dims, const void* w_packed, const void* x_in,
                              void* x_out, int32_t total_rows_ub, const int32_t* cu_seqlens,
                              const int32_t* seqused, int32_t batch, float act_eps,
                              int32_t* act_count, void* workspace, size_t workspace_bytes,
                              hipStream_t stream, hipEvent_t* ev, const void* kv_cache = nullptr,
                              const int32_t* cu_kv = nullptr, bool own_status = false,
                              int32_t* status = nullptr, const DetectStep* det = nullptr) {
  int rc = check_dims(dims);
  if (rc) return rc;
  if (!w_packed || !x_in || !x_out || !cu_seqlens || !workspace)
    return fail(SEER_EINVAL, "a required pointer is NULL");
  if (batch < 1) return fail(SEER_EINVAL, "batch must be >= 1 (got %d)", batch);
  if (total_rows_ub < 1) return fail(SEER_EINVAL, "total_rows_ub must be >= 1 (got %d)", total_rows_ub);
  if (x_in == x_out) return fail(SEER_EINVAL, "x_in and x_out may not alias");
  if (act_count && !(act_eps >= 0.0f)) return fail(SEER_EINVAL, "act_eps must be >= 0");
  const bool bf16 = dims->dtype == SEER_DTYPE_BF16;
  if (bf16 && (!aligned(w_packed, 256) || !aligned(x_in, 16) || !aligned(x_out, 16)))
    return fail(SEER_EINVAL, "bf16 weights need 256-byte and rows 16-byte alignment");
  if (!aligned(workspace, 256)) return fail(SEER_EINVAL, "workspace must be 256-byte aligned");
  if (bf16) {
    // the bf16 kernels address rows with 32-bit byte offsets: the widest row
    // buffer (qkv, 3 d, or the activations, d_ff) must stay below 4 GiB
    const size_t wide = (size_t)(3 * dims->d_model > dims->d_ff ? 3 * dims->d_model : dims->d_ff);
    if ((size_t)total_rows_ub * wide * 2 >= ((size_t)1 << 32))
      return fail(SEER_EUNSUPPORTED, "total_rows_ub %d too large for the bf16 kernels (rows x %zu bf16 >= 4 GiB)",
                  total_rows_ub, wide);
  }
  const WsLayout L = ws_layout(dims, total_rows_ub);
  if (workspace_bytes < L.total)
    return fail(SEER_EWORKSPACE, "workspace holds %zu bytes, need %zu", workspace_bytes, L.total);

  const int d = dims->d_model, I = dims->d_ff, R = total_rows_ub;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  void* qkv = ws + L.qkv;
  void* o = ws + L.o;
  void* h1 = ws + L.h1;
  void* act = ws + L.act;
  float* inv1 = reinterpret_cast<float*>(ws + L.inv1);
  float* inv2 = reinterpret_cast<float*>(ws + L.inv2);
  void* h1lo = ws + L.h1lo;
  const bool rope = dims->rope_theta > 0.0f;
  int* rpos = reinterpret_cast<int*>(ws + L.pos);
  double* rfreq = reinterpret_cast<double*>(ws + L.freq);
  float* part = L.part_bytes ? reinterpret_cast<float*>(ws + L.part) : nullptr;
  int n_units = 0;                      // CUs: sizes the split of a partly filled last GEMM round
  if (bf16) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_units, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return hip_fail("device query");
  }
  const int* m_ptr = cu_seqlens + batch;
  const seer::PackedLayout P = seer::packed_layout(d, I, bf16);
  const size_t es = bf16 ? 2 : 4;
  const uint8_t* wb = static_cast<const uint8_t*>(w_packed);
  auto gemm = bf16 ? seer::launch_gemm_bf16 : seer::launch_gemm_f32;

  // a NULL entry skips that mark: each record on the stream delays the next
  // launch by a few microseconds, so a caller timing one kernel passes only
  // the two events around it
  auto mark = [&](int k) { return ev && ev[k] ? hipEventRecord(ev[k], stream) : hipSuccess; };
  if (mark(0) != hipSuccess) return hip_fail("event record");
  // 1. RMSNorm statistics of the layer input (+ rotary positions)
  {
    seer::RopeArgs ra{};
    ra.cu = cu_seqlens; ra.B = batch; ra.cu_kv = cu_kv; ra.pos = rpos; ra.freq = rfreq;
    ra.theta = dims->rope_theta; ra.head_dim = dims->head_dim;
    if (seer::launch_rms_inv(bf16, x_in, d, d, m_ptr, R, dims->rms_eps, inv1, stream, rope ? &ra : nullptr))
      return hip_fail("rms launch");
  }
  // 2. QKV projection, RMSNorm folded in as a row scale
  if (mark(1) != hipSuccess) return hip_fail("event record");
  {
    seer::GemmParams g{};
    g.n_units = n_units;
    g.partial = part; g.partial_bytes = L.part_bytes;
    g.A = x_in; g.B = wb + P.qkv * es; g.C = qkv; g.rs = inv1;
    g.m_ptr = m_ptr; g.m_ub = R; g.N = 3 * d; g.K = d;
    g.lda = d; g.ldb = d; g.ldc = 3 * d;
    g.f16_col0 = bf16 ? 2 * d : 0;     // V goes to the attention's fp16 PV product
    // V beyond fp16 range is reported in the workspace status word (or in the
    // caller's word, for the no-allocation entry point)
    g.status = !bf16 ? nullptr : own_status ? status : reinterpret_cast<int*>(ws);
    g.perm_col1 = bf16 ? 2 * d : 0;    // q and k rows are packed head-permuted
    if (rope && bf16) {
      // q and k rotated in the epilogue, where each lane holds rotary pairs
      g.rope_pos = rpos; g.rope_freq = rfreq; g.rope_col1 = 2 * d;
    }
    if (gemm(rope && bf16 ? seer::EPI_SCALE_ROPE : seer::EPI_SCALE, g, stream)) return hip_fail("qkv gemm launch");
    if (rope && !bf16 &&
        seer::launch_rope_f32(static_cast<float*>(qkv), d, dims->n_heads, dims->head_dim, m_ptr, R, rpos, rfreq,
                              stream))
      return hip_fail("rope launch");
  }
  // 3. bidirectional varlen attention
  if (mark(2) != hipSuccess) return hip_fail("event record");
  {
    seer::AttnParams a{};
    a.qkv = qkv; a.out = o; a.cu = cu_seqlens; a.used = seqused; a.B = batch;
    a.d = d; a.n_heads = dims->n_heads; a.head_dim = dims->head_dim; a.rows_ub = R;
    a.scale = 1.0f / sqrtf((float)dims->head_dim);
    a.kv = kv_cache; a.cu_kv = cu_kv;
    if ((bf16 ? seer::launch_attn_bf16(a, stream) : seer::launch_attn_f32(a, stream)))
      return hip_fail("attention launch");
  }
  // 4. output projection + residual
  if (mark(3) != hipSuccess) return hip_fail("event record");
  {
    seer::GemmParams g{};
    g.n_units = n_units;
    g.partial = part; g.partial_bytes = L.part_bytes;
    g.A = o; g.B = wb + P.o * es; g.C = h1; g.R = x_in; g.C2 = h1lo;
    g.m_ptr = m_ptr; g.m_ub = R; g.N = d; g.K = d;
    g.lda = d; g.ldb = d; g.ldc = d; g.ldr = d;
    if (gemm(bf16 ? seer::EPI_RESID_SPLIT : seer::EPI_RESID, g, stream)) return hip_fail("o gemm launch");
  }
  // 5. RMSNorm statistics before the MLP
  if (mark(4) != hipSuccess) return hip_fail("event record");
  if (seer::launch_rms_inv(bf16, h1, d, d, m_ptr, R, dims->rms_eps, inv2, stream))
    return hip_fail("rms launch");
  // 6. gate/up projection + SwiGLU (+ near-zero count)
  {
    if (act_count && seer::launch_zero_i32(act_count, R, stream)) return hip_fail("zero launch");
    seer::GemmParams g{};
    g.n_units = n_units;
    g.partial = part; g.partial_bytes = L.part_bytes;
    g.A = h1; g.C = act; g.rs = inv2; g.cnt = act_count; g.eps = act_eps;
    g.m_ptr = m_ptr; g.m_ub = R; g.K = d; g.lda = d; g.ldb = d; g.ldc = I;
    if (bf16) {
      g.B = wb + P.gu * es;
      g.N = 2 * I;
    } else {
      g.B = wb + P.gu * es;
      g.B2 = wb + (P.gu + (size_t)I * d) * es;
      g.N = I;
    }
    if (mark(5) != hipSuccess) return hip_fail("event record");
    if (gemm(act_count ? seer::EPI_SWIGLU_COUNT : seer::EPI_SWIGLU, g, stream))
      return hip_fail("gate/up gemm launch");
  }
  // 6b. (detection layer) the SNR scan on the counts, and the row tiles that
  // hold kept rows: the down projection computes only those
  int* tmap = nullptr;
  if (det) {
    if (mark(6) != hipSuccess) return hip_fail("event record");
    seer::DetectParams dp{};
    dp.cnt = act_count; dp.cu = cu_seqlens; dp.win_off = det->win_off; dp.win_len = det->win_len;
    dp.B = batch; dp.d_ff = I;
    dp.tau_num = det->snr->tau_num; dp.tau_den = det->snr->tau_den;
    dp.gamma_num = det->snr->gamma_num; dp.gamma_den = det->snr->gamma_den;
    dp.lookahead = det->snr->lookahead;
    dp.boundary = det->boundary; dp.keep_len = det->keep_len;
    if (seer::launch_detect(dp, stream)) return hip_fail("detect launch");
    if (bf16) {
      tmap = reinterpret_cast<int*>(ws + L.tmap);
      seer::KeptTilesParams kp{};
      kp.cu = cu_seqlens; kp.win_off = det->win_off; kp.win_len = det->win_len; kp.keep_len = det->keep_len;
      kp.B = batch; kp.rows_ub = R; kp.map = tmap;
      if (seer::launch_kept_tiles(kp, stream)) return hip_fail("kept tiles launch");
    }
  }
  const int e_down = det ? 7 : 6;
  // 7. down projection + residual
  if (mark(e_down) != hipSuccess) return hip_fail("event record");
  {
    seer::GemmParams g{};
    g.n_units = n_units;
    g.partial = part; g.partial_bytes = L.part_bytes;
    g.A = act; g.B = wb + P.dn * es; g.C = x_out; g.R = h1; g.R2 = h1lo;
    g.m_ptr = m_ptr; g.m_ub = R; g.N = d; g.K = I;
    g.lda = I; g.ldb = I; g.ldc = d; g.ldr = d;
    g.mtiles = tmap;
    if (gemm(bf16 ? seer::EPI_RESID_PAIR : seer::EPI_RESID, g, stream)) return hip_fail("down gemm launch");
  }
  if (mark(e_down + 1) != hipSuccess) return hip_fail("event record");
  return ok();
}

static int layer_detect_impl(const seer_dims* dims, const void* w_packed, const void* x_in, void* x_out,
                             int32_t total_rows_ub, const int32_t* cu_seqlens, int32_t batch, float act_eps,
                             int32_t* act_count, const int32_t* win_off, const int32_t* win_len,
                             const seer_snr_params* params, int32_t* boundary, int32_t* keep_len,
                             void* workspace, size_t workspace_bytes, hipStream_t stream, hipEvent_t* ev) {
  if (!act_count || !win_off || !win_len || !params || !boundary || !keep_len)
    return fail(SEER_EINVAL, "a required pointer is NULL");
  int rc = check_snr(params);
  if (rc) return rc;
  const DetectStep det{win_off, win_len, params, boundary, keep_len};
  return layer_forward_impl(dims, w_packed, x_in, x_out, total_rows_ub, cu_seqlens, nullptr, batch, act_eps,
                            act_count, workspace, workspace_bytes, stream, ev, nullptr, nullptr, false, nullptr,
                            &det);
}

int seer_layer_forward_detect(const seer_dims* dims, const void* w_packed, const void* x_in, void* x_out,
                              int32_t total_rows_ub, const int32_t* cu_seqlens, int32_t batch, float act_eps,
                              int32_t* act_count, const int32_t* win_off, const int32_t* win_len,
                              const seer_snr_params* params, int32_t* boundary, int32_t* keep_len,
                              void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return layer_detect_impl(dims, w_packed, x_in, x_out, total_rows_ub, cu_seqlens, batch, act_eps, act_count,
                           win_off, win_len, params, boundary, keep_len, workspace, workspace_bytes, stream,
                           nullptr);
}

int seer_layer_forward_detect_timed(const seer_dims* dims, const void* w_packed, const void* x_in, void* x_out,
                                    int32_t total_rows_ub, const int32_t* cu_seqlens, int32_t batch,
                                    float act_eps, int32_t* act_count, const int32_t* win_off,
                                    const int32_t* win_len, const seer_snr_params* params, int32_t* boundary,
                                    int32_t* keep_len, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream, hipEvent_t* events) {
  if (!events) return fail(SEER_EINVAL, "events is NULL");
  return layer_detect_impl(dims, w_packed, x_in, x_out, total_rows_ub, cu_seqlens, batch, act_eps, act_count,
                           win_off, win_len, params, boundary, keep_len, workspace, workspace_bytes, stream,
                           events);
}

int seer_layer_forward_varlen(const seer_dims* dims, const void* w_packed, const void* x_in,
                              void* x_out, int32_t total_rows_ub, const int32_t* cu_seqlens,
                              const int32_t* seqused, int32_t batch, float act_eps,
                              int32_t* act_count, void* workspace, size_t workspace_bytes,
                              hipStream_t stream) {
  return layer_forward_impl(dims, w_packed, x_in, x_out, total_rows_ub, cu_seqlens, seqused, batch,
                            act_eps, act_count, workspace, workspace_bytes, stream, nullptr);
}

}  // extern "C"

// ---- the layer without allocation ------------------------------------------
// A workspace that lives in the library, for callers that cannot allocate:
// one copy of this array per GPU, held until the process ends.  Host code
// never uses the array's name as an address: its device address is looked up
// once per device (hipGetSymbolAddress) and kept in scratch_ptr.
static constexpr size_t kScratchBytes = (size_t)256 << 20;
static __device__ __attribute__((aligned(256))) uint8_t scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_of_current_device(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return hip_fail("hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(SEER_EUNSUPPORTED, "device %d beyond the %d supported", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(SEER_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SEER_OK;
}
}  // namespace

extern "C" {

int seer_layer_forward_varlen_noalloc(const seer_dims* dims, const void* w_packed, const void* x_in,
                                      void* x_out, int32_t total_rows_ub, const int32_t* cu_seqlens,
                                      const int32_t* seqused, int32_t batch, float act_eps,
                                      int32_t* act_count, int32_t* status, hipStream_t stream) {
  int rc = check_dims(dims);
  if (rc) return rc;
  if (total_rows_ub < 1) return fail(SEER_EINVAL, "total_rows_ub must be >= 1 (got %d)", total_rows_ub);
  const size_t need = ws_layout(dims, total_rows_ub).total;
  if (need > kScratchBytes)
    return fail(SEER_EWORKSPACE,
                "total_rows_ub %d needs %zu bytes of workspace; the no-allocation entry point has %zu "
                "(seer_layer_workspace_bytes gives the need per rows bound)", total_rows_ub, need, kScratchBytes);
  void* ws = nullptr;
  rc = scratch_of_current_device(&ws);
  if (rc) return rc;
  return layer_forward_impl(dims, w_packed, x_in, x_out, total_rows_ub, cu_seqlens, seqused, batch, act_eps,
                            act_count, ws, kScratchBytes, stream, nullptr, nullptr, nullptr, true, status);
}

int seer_layer_forward_varlen_timed(const seer_dims* dims, const void* w_packed, const void* x_in,
                                    void* x_out, int32_t total_rows_ub, const int32_t* cu_seqlens,
                                    const int32_t* seqused, int32_t batch, float act_eps,
                                    int32_t* act_count, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream, hipEvent_t* events) {
  if (!events) return fail(SEER_EINVAL, "events is NULL");
  return layer_forward_impl(dims, w_packed, x_in, x_out, total_rows_ub, cu_seqlens, seqused, batch,
                            act_eps, act_count, workspace, workspace_bytes, stream, events);
}

int seer_layer_forward_cached(const seer_dims* dims, const void* w_packed, const void* x_in,
                              void* x_out, int32_t total_rows_ub, const int32_t* cu_seqlens,
                              const int32_t* seqused, int32_t batch, const void* kv_cache,
                              const int32_t* cu_kv, int32_t kv_rows_ub, void* workspace,
                              size_t workspace_bytes, hipStream_t stream) {
  int rc = check_dims(dims);
  if (rc) return rc;
  if (!kv_cache || !cu_kv) return fail(SEER_EINVAL, "kv_cache/cu_kv is NULL");
  if (kv_rows_ub < 0) return fail(SEER_EINVAL, "kv_rows_ub must be >= 0");
  if (!aligned(kv_cache, 16)) return fail(SEER_EINVAL, "kv_cache must be 16-byte aligned");
  if ((size_t)kv_rows_ub * 2 * (size_t)dims->d_model >= ((size_t)1 << 32))
    return fail(SEER_EUNSUPPORTED, "kv_rows_ub %d is too large: cache element offsets must fit 32 bits", kv_rows_ub);
  return layer_forward_impl(dims, w_packed, x_in, x_out, total_rows_ub, cu_seqlens, seqused, batch, 0.0f,
                            nullptr, workspace, workspace_bytes, stream, nullptr, kv_cache, cu_kv);
}

int seer_kv_export(const seer_dims* dims, const void* workspace, size_t workspace_bytes,
                   int32_t total_rows_ub, const int32_t* cu_seqlens, int32_t batch,
                   const int32_t* cu_kv, int32_t kv_rows_ub, void* kv_dst, hipStream_t stream) {
  int rc = check_dims(dims);
  if (rc) return rc;
  if (!workspace || !cu_seqlens || !cu_kv || !kv_dst) return fail(SEER_EINVAL, "a required pointer is NULL");
  if (batch < 1) return fail(SEER_EINVAL, "batch must be >= 1 (got %d)", batch);
  if (total_rows_ub < 1) return fail(SEER_EINVAL, "total_rows_ub must be >= 1 (got %d)", total_rows_ub);
  if (kv_rows_ub < 0) return fail(SEER_EINVAL, "kv_rows_ub must be >= 0");
  if (!aligned(workspace, 256) || !aligned(kv_dst, 16)) return fail(SEER_EINVAL, "misaligned workspace or kv_dst");
  const WsLayout L = ws_layout(dims, total_rows_ub);
  if (workspace_bytes < L.total)
    return fail(SEER_EWORKSPACE, "workspace holds %zu bytes, need %zu", workspace_bytes, L.total);
  seer::KvExportParams p{};
  p.qkv = static_cast<const uint8_t*>(workspace) + L.qkv;
  p.cu = cu_seqlens; p.cu_kv = cu_kv; p.dst = static_cast<uint8_t*>(kv_dst);
  p.B = batch; p.d = dims->d_model; p.es = dims->dtype == SEER_DTYPE_BF16 ? 2 : 4;
  p.rows_ub = total_rows_ub;
  if (seer::launch_kv_export(p, kv_rows_ub, stream)) return hip_fail("kv export launch");
  return ok();
}

int seer_step0_detect(const int32_t* act_count, const int32_t* cu_seqlens, const int32_t* win_off,
                      const int32_t* win_len, int32_t batch, int32_t d_ff,
                      const seer_snr_params* params, int32_t* boundary, int32_t* keep_len,
                      hipStream_t stream) {
  if (!act_count || !cu_seqlens || !win_off || !win_len || !params || !boundary || !keep_len)
    return fail(SEER_EINVAL, "a required pointer is NULL");
  if (batch < 1) return fail(SEER_EINVAL, "batch must be >= 1 (got %d)", batch);
  if (d_ff < 1) return fail(SEER_EINVAL, "d_ff must be >= 1");
  int rc = check_snr(params);
  if (rc) return rc;
  seer::DetectParams p{};
  p.cnt = act_count; p.cu = cu_seqlens; p.win_off = win_off; p.win_len = win_len;
  p.B = batch; p.d_ff = d_ff;
  p.tau_num = params->tau_num; p.tau_den = params->tau_den;
  p.gamma_num = params->gamma_num; p.gamma_den = params->gamma_den;
  p.lookahead = params->lookahead;
  p.boundary = boundary; p.keep_len = keep_len;
  if (seer::launch_detect(p, stream)) return hip_fail("detect launch");
  return ok();
}

int seer_batch_repack(const seer_repack_desc* desc, const void* const* src, void* const* dst,
                      int32_t n_buffers, const int32_t* cu_src, const int32_t* win_off,
                      const int32_t* win_len, const int32_t* keep_len, int32_t batch,
                      int32_t* cu_dst, int32_t* seqused, int32_t* route, seer_route_ctrl* ctrl_dev,
                      seer_route_ctrl* ctrl_host, hipStream_t stream) {
  if (!desc || !src || !dst || !cu_src || !win_off || !win_len || !keep_len || !cu_dst || !seqused ||
      !route)
    return fail(SEER_EINVAL, "a required pointer is NULL");
  if (batch < 1 || batch > seer::kRepackMaxBatch)
    return fail(batch < 1 ? SEER_EINVAL : SEER_EUNSUPPORTED, "batch must be in [1, %d] (got %d)",
                seer::kRepackMaxBatch, batch);
  if (n_buffers < 1 || n_buffers > seer::kRepackMaxBuffers)
    return fail(SEER_EINVAL, "n_buffers must be in [1, %d]", seer::kRepackMaxBuffers);
  if (desc->policy < 0 || desc->policy > 2) return fail(SEER_EINVAL, "unknown policy %d", desc->policy);
  if (desc->tau_pad_den < 1 || desc->tau_pad_num < 0) return fail(SEER_EINVAL, "bad tau_pad");
  if (desc->granule < 1) return fail(SEER_EINVAL, "granule must be >= 1");
  if (desc->row_bytes < 16 || desc->row_bytes % 16) return fail(SEER_EINVAL, "row_bytes must be a positive multiple of 16");
  if (desc->dst_capacity_rows < 0) return fail(SEER_EINVAL, "dst_capacity_rows must be >= 0");
  seer::RepackParams p{};
  for (int i = 0; i < n_buffers; ++i) {
    if (!src[i] || !dst[i]) return fail(SEER_EINVAL, "buffer %d is NULL", i);
    if (!aligned(src[i], 16) || !aligned(dst[i], 16)) return fail(SEER_EINVAL, "buffers must be 16-byte aligned");
    if (src[i] == dst[i]) return fail(SEER_EINVAL, "src and dst may not alias");
    p.src[i] = static_cast<const uint8_t*>(src[i]);
    p.dst[i] = static_cast<uint8_t*>(dst[i]);
  }
  p.n_buffers = n_buffers;
  p.cu_src = cu_src; p.win_off = win_off; p.win_len = win_len; p.keep_len = keep_len;
  p.B = batch; p.policy = desc->policy;
  p.tau_num = desc->tau_pad_num; p.tau_den = desc->tau_pad_den;
  p.granule = desc->granule; p.row_bytes = desc->row_bytes;
  p.dst_capacity_rows = desc->dst_capacity_rows;
  p.cu_dst = cu_dst; p.seqused = seqused; p.route = route;
  p.window_only = (desc->flags & SEER_REPACK_WINDOW_ONLY) != 0;
  p.ctrl_dev = reinterpret_cast<int*>(ctrl_dev);
  p.ctrl_host = reinterpret_cast<int*>(ctrl_host);
  if (seer::launch_repack(p, stream)) return hip_fail("repack launch");
  return ok();
}

// ---- synthetic LM head and remasking sampler --------------------------------

static size_t lm_partials_offset(int32_t rows_ub) { return up256((size_t)rows_ub * 4); }

size_t seer_lm_head_workspace_bytes(const seer_dims* dims, int32_t vocab, int32_t rows_ub) {
  if (check_dims(dims) != SEER_OK || vocab <= 0 || rows_ub < 0) return 0;
  return lm_partials_offset(rows_ub) + up256((size_t)rows_ub * (size_t)(vocab / 64) * sizeof(seer::ArgmaxPartial));
}

// shape checks shared by the head's two calls
static int check_head(const seer_dims* dims, int32_t vocab, const char* what) {
  int rc = check_dims(dims);
  if (rc) return rc;
  if (dims->dtype != SEER_DTYPE_BF16) return fail(SEER_EUNSUPPORTED, "the LM head runs on bf16 layers only");
  if (vocab <= 0 || vocab % 256 != 0) return fail(SEER_EUNSUPPORTED, "vocab must be a positive multiple of 256 (got %d)", vocab);
  // the GEMM addresses its operands with 32-bit byte offsets
  if ((size_t)vocab * dims->d_model * 2 >= ((size_t)1 << 32))
    return fail(SEER_EUNSUPPORTED, "%s must stay below 4 GiB", what);
  return SEER_OK;
}

int seer_lm_head_prepack(const seer_dims* dims, const void* w_lm, int32_t vocab, void* dst, size_t dst_bytes,
                         hipStream_t stream) {
  int rc = check_head(dims, vocab, "w_lm");
  if (rc) return rc;
  if (!w_lm || !dst) return fail(SEER_EINVAL, "w_lm/dst is NULL");
  if (!aligned(w_lm, 16) || !aligned(dst, 256)) return fail(SEER_EINVAL, "w_lm needs 16-byte, dst 256-byte alignment");
  const size_t need = (size_t)vocab * dims->d_model * 2;
  if (dst_bytes < need) return fail(SEER_EINVAL, "dst holds %zu bytes, need %zu", dst_bytes, need);
  if (seer::launch_pack_frag(w_lm, vocab, dims->d_model, dst, stream)) return hip_fail("pack launch");
  return ok();
}

int seer_lm_head_predict(const seer_dims* dims, const void* w_packed, int32_t vocab, const void* x, int32_t rows_ub,
                         const int32_t* cu_seqlens, int32_t batch, int32_t* pred, float* conf, void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
  int rc = check_head(dims, vocab, "the packed head weight");
  if (rc) return rc;
  if (!w_packed || !x || !cu_seqlens || !pred || !conf || !workspace)
    return fail(SEER_EINVAL, "a required pointer is NULL");
  if (batch < 1 || rows_ub < 1) return fail(SEER_EINVAL, "batch and rows_ub must be >= 1");
  if ((size_t)rows_ub * dims->d_model * 2 >= ((size_t)1 << 32)) return fail(SEER_EUNSUPPORTED, "x must stay below 4 GiB");
  if (!aligned(w_packed, 16) || !aligned(x, 16) || !aligned(workspace, 256))
    return fail(SEER_EINVAL, "w_packed and x need 16-byte, workspace 256-byte alignment");
  const size_t need = seer_lm_head_workspace_bytes(dims, vocab, rows_ub);
  if (workspace_bytes < need) return fail(SEER_EWORKSPACE, "workspace holds %zu bytes, need %zu", workspace_bytes, need);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  float* inv = reinterpret_cast<float*>(ws);
  void* part = ws + lm_partials_offset(rows_ub);
  const int* m_ptr = cu_seqlens + batch;
  const int d = dims->d_model;
  if (seer::launch_rms_inv(true, x, d, d, m_ptr, rows_ub, dims->rms_eps, inv, stream)) return hip_fail("rms launch");
  seer::GemmParams g{};
  g.A = x; g.B = w_packed; g.C = part; g.rs = inv;
  g.m_ptr = m_ptr; g.m_ub = rows_ub; g.N = vocab; g.K = d;
  g.lda = d; g.ldb = d; g.ldc = vocab / 64;   // one partial per row and 64 columns
  g.n_units = 0;
  if (seer::launch_gemm_bf16(seer::EPI_ARGMAX, g, stream)) return hip_fail("lm head gemm launch");
  if (seer::launch_argmax_reduce(part, vocab / 64, m_ptr, rows_ub, pred, conf, stream))
    return hip_fail("argmax reduce launch");
  return ok();
}

int seer_remask_step(const seer_dims* dims, const int32_t* cu_seqlens, const int32_t* seqused, int32_t batch,
                     int32_t max_used, int32_t steps_left, const int32_t* pred, const float* conf, int32_t* tokens,
                     const void* x0, const void* emb, int32_t vocab, void* x_next, hipStream_t stream) {
  int rc = check_dims(dims);
  if (rc) return rc;
  if (dims->dtype != SEER_DTYPE_BF16) return fail(SEER_EUNSUPPORTED, "the sampler runs on bf16 layers only");
  if (!cu_seqlens || !pred || !conf || !tokens || !x0 || !emb || !x_next)
    return fail(SEER_EINVAL, "a required pointer is NULL");
  if (batch < 1 || vocab < 1 || steps_left < 1) return fail(SEER_EINVAL, "batch, vocab and steps_left must be >= 1");
  if (max_used < 0 || max_used > 8192) return fail(SEER_EUNSUPPORTED, "max_used must be in [0, 8192] (got %d)", max_used);
  if (!aligned(x0, 16) || !aligned(emb, 16) || !aligned(x_next, 16)) return fail(SEER_EINVAL, "rows need 16-byte alignment");
  seer::RemaskParams p{};
  p.cu = cu_seqlens; p.used = seqused; p.B = batch; p.max_used = max_used; p.steps_left = steps_left;
  p.pred = pred; p.conf = conf; p.tokens = tokens;
  p.x0 = static_cast<const uint16_t*>(x0); p.emb = static_cast<const uint16_t*>(emb); p.vocab = vocab;
  p.x_next = static_cast<uint16_t*>(x_next); p.d = dims->d_model;
  if (seer::launch_remask(p, stream)) return hip_fail("remask launch");
  return ok();
}

// ---- recorded launch sequences (Sec. 3.5, graph-compatible paths) ----------

struct seer_graph_ {
  hipGraph_t graph;
  hipGraphExec_t exec;
};

int seer_graph_begin(hipStream_t stream) {
  if (stream == nullptr) return fail(SEER_EINVAL, "the default (null) stream cannot be recorded; use a created stream");
  hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &st) != hipSuccess) return hip_fail("hipStreamIsCapturing");
  if (st != hipStreamCaptureStatusNone) return fail(SEER_EINVAL, "the stream is already being recorded");
  if (hipStreamBeginCapture(stream, hipStreamCaptureModeThreadLocal) != hipSuccess)
    return hip_fail("hipStreamBeginCapture");
  return ok();
}

int seer_graph_end(hipStream_t stream, seer_graph_t* graph) {
  if (graph == nullptr) return fail(SEER_EINVAL, "graph is NULL");
  *graph = nullptr;
  if (stream == nullptr) return fail(SEER_EINVAL, "stream is NULL");
  hipGraph_t g = nullptr;
  if (hipStreamEndCapture(stream, &g) != hipSuccess || g == nullptr) {
    if (g) (void)hipGraphDestroy(g);
    return hip_fail("hipStreamEndCapture (a call recorded since seer_graph_begin failed, or the stream "
                    "was not being recorded)");
  }
  hipGraphExec_t exec = nullptr;
  if (hipGraphInstantiate(&exec, g, nullptr, nullptr, 0) != hipSuccess) {
    (void)hipGraphDestroy(g);
    return hip_fail("hipGraphInstantiate");
  }
  *graph = new seer_graph_{g, exec};
  return ok();
}

int seer_graph_launch(seer_graph_t graph, hipStream_t stream) {
  if (graph == nullptr) return fail(SEER_EINVAL, "graph is NULL");
  if (hipGraphLaunch(graph->exec, stream) != hipSuccess) return hip_fail("hipGraphLaunch");
  return ok();
}

int seer_graph_destroy(seer_graph_t graph) {
  if (graph == nullptr) return ok();
  const bool bad = hipGraphExecDestroy(graph->exec) != hipSuccess;
  const bool bad2 = hipGraphDestroy(graph->graph) != hipSuccess;
  delete graph;
  if (bad || bad2) return hip_fail("hipGraphExecDestroy / hipGraphDestroy");
  return ok();
}

}  // extern "C"
