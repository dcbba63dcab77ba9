// fp32 variants of the layer kernels (any d_model, d_ff; head_dim <= 128).
//
// These serve the small fp32 layer shape; they are plain vector-ALU kernels
// (LDS-tiled GEMM with the same fused epilogues as the bf16 path, and a
// one-query-per-lane online-softmax attention) and are not performance
// critical.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace seer {

namespace {
constexpr int TM = 64, TN = 64, TK = 16;
}

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmParams p) {
  constexpr bool kGlu = (EPI == EPI_SWIGLU || EPI == EPI_SWIGLU_COUNT);
  __shared__ float As[TK][TM + 4];
  __shared__ float Bs[TK][TN + 4];
  __shared__ float B2s[kGlu ? TK : 1][TN + 4];
  const int M = rows_from(p.m_ptr, p.m_ub);
  const int m0 = blockIdx.y * TM;
  const int n0 = blockIdx.x * TN;
  if (m0 >= M) return;
  const float* A = static_cast<const float*>(p.A);
  const float* Bm = static_cast<const float*>(p.B);
  const float* B2 = static_cast<const float*>(p.B2);
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  float acc[4][4], acc2[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) { acc[i][j] = 0.0f; acc2[i][j] = 0.0f; }

  for (int k0 = 0; k0 < p.K; k0 += TK) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = tid + 256 * i;
      const int r = e >> 4, kk = e & 15;
      const int gk = k0 + kk;
      const int gr = m0 + r, gn = n0 + r;
      As[kk][r] = (gr < M && gk < p.K) ? A[(size_t)gr * p.lda + gk] : 0.0f;
      Bs[kk][r] = (gn < p.N && gk < p.K) ? Bm[(size_t)gn * p.ldb + gk] : 0.0f;
      if constexpr (kGlu) B2s[kk][r] = (gn < p.N && gk < p.K) ? B2[(size_t)gn * p.ldb + gk] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], b[4], b2[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        b[j] = Bs[kk][tx * 4 + j];
        if constexpr (kGlu) b2[j] = B2s[kk][tx * 4 + j];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
          if constexpr (kGlu) acc2[i][j] = fmaf(a[i], b2[j], acc2[i][j]);
        }
    }
    __syncthreads();
  }

  float* C = static_cast<float*>(p.C);
  const float* R = static_cast<const float*>(p.R);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= M) continue;
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx * 4 + j;
      if (col >= p.N) continue;
      float v;
      if constexpr (EPI == EPI_SCALE) {
        v = acc[i][j] * p.rs[row];
      } else if constexpr (EPI == EPI_RESID) {
        v = R[(size_t)row * p.ldr + col] + acc[i][j];
      } else {
        const float s = p.rs[row];
        v = silu(acc[i][j] * s) * (acc2[i][j] * s);
        cnt += fabsf(v) < p.eps ? 1 : 0;
      }
      C[(size_t)row * p.ldc + col] = v;
    }
    if constexpr (EPI == EPI_SWIGLU_COUNT) {
      if (cnt) atomicAdd(p.cnt + row, cnt);
    }
  }
}

int launch_gemm_f32(int epi, const GemmParams& p, hipStream_t s) {
  dim3 grid((p.N + TN - 1) / TN, (p.m_ub + TM - 1) / TM), block(256);
  switch (epi) {
    case EPI_SCALE: hipLaunchKernelGGL(gemm_f32_kernel<EPI_SCALE>, grid, block, 0, s, p); break;
    case EPI_RESID: hipLaunchKernelGGL(gemm_f32_kernel<EPI_RESID>, grid, block, 0, s, p); break;
    case EPI_SWIGLU: hipLaunchKernelGGL(gemm_f32_kernel<EPI_SWIGLU>, grid, block, 0, s, p); break;
    case EPI_SWIGLU_COUNT:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_SWIGLU_COUNT>, grid, block, 0, s, p); break;
    default: return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ---------------------------------------------------------------------------
// fp32 attention: one query per lane, 64 queries per workgroup, keys staged in
// LDS 32 at a time, online softmax per query.
namespace {
constexpr int AQ = 64;
constexpr int AK = 32;
}

template <int DH>
__global__ __launch_bounds__(AQ) void attn_f32_kernel(AttnParams p) {
  __shared__ float ks[AK][DH];
  __shared__ float vs[AK][DH];
  int b = -1, t = 0;
  {
    int acc = 0;
    for (int s = 0; s < p.B; ++s) {
      int len = p.cu[s + 1] - p.cu[s];
      len = len < 0 ? 0 : len;
      const int nt = (len + AQ - 1) / AQ;
      if ((int)blockIdx.x < acc + nt) { b = s; t = blockIdx.x - acc; break; }
      acc += nt;
    }
  }
  if (b < 0) return;
  const int h = blockIdx.y;
  const int s0 = p.cu[b];
  if (s0 < 0 || s0 >= p.rows_ub) return;
  int len = p.cu[b + 1] - s0;
  len = len > p.rows_ub - s0 ? p.rows_ub - s0 : len;
  if (t * AQ >= len) return;
  int used = p.used ? p.used[b] : len;
  used = used < 0 ? 0 : (used > len ? len : used);
  const float* qkv = static_cast<const float*>(p.qkv);
  float* out = static_cast<float*>(p.out);
  const size_t ld = (size_t)3 * p.d;
  const int q_row = t * AQ + threadIdx.x;
  const int q_src = q_row < len ? q_row : len - 1;
  float q[DH], o[DH];
#pragma unroll
  for (int e = 0; e < DH; ++e) {
    q[e] = e < p.head_dim ? qkv[(size_t)(s0 + q_src) * ld + h * p.head_dim + e] * p.scale : 0.0f;
    o[e] = 0.0f;
  }
  // keys: the cached prefix rows (if any), then the sequence's own used rows
  int P = 0, kv0 = 0;
  if (p.cu_kv) {
    kv0 = p.cu_kv[b];
    P = p.cu_kv[b + 1] - kv0;
    P = P < 0 ? 0 : P;
  }
  const int n_keys = P + used;
  const float* kvc = static_cast<const float*>(p.kv);
  float m = -INFINITY, l = 0.0f;
  for (int k0 = 0; k0 < n_keys; k0 += AK) {
    for (int e = threadIdx.x; e < AK * DH; e += AQ) {
      const int kk = e / DH, c = e % DH;
      const int key = k0 + kk;
      const bool ok = key < n_keys && c < p.head_dim;
      const float* kr = !ok ? nullptr
          : key < P ? kvc + (size_t)(kv0 + key) * 2 * p.d + h * p.head_dim + c
                    : qkv + (size_t)(s0 + key - P) * ld + p.d + h * p.head_dim + c;
      ks[kk][c] = ok ? kr[0] : 0.0f;
      vs[kk][c] = ok ? kr[p.d] : 0.0f;
    }
    __syncthreads();
    const int nk = min(AK, n_keys - k0);
    for (int kk = 0; kk < nk; ++kk) {
      float sc = 0.0f;
#pragma unroll
      for (int e = 0; e < DH; ++e) sc = fmaf(q[e], ks[kk][e], sc);
      const float mn = fmaxf(m, sc);
      const float alpha = __expf(m - mn);
      const float pe = __expf(sc - mn);
      l = l * alpha + pe;
#pragma unroll
      for (int e = 0; e < DH; ++e) o[e] = fmaf(pe, vs[kk][e], o[e] * alpha);
      m = mn;
    }
    __syncthreads();
  }
  if (q_row < len) {
    const float inv = (q_row < used && l > 0.0f) ? 1.0f / l : 0.0f;
    for (int e = 0; e < p.head_dim; ++e)
      out[(size_t)(s0 + q_row) * p.d + h * p.head_dim + e] = o[e] * inv;
  }
}

int launch_attn_f32(const AttnParams& p, hipStream_t s) {
  if (p.cu_kv && !p.kv) return -1;
  dim3 grid((p.rows_ub + AQ - 1) / AQ + p.B, p.n_heads), block(AQ);
  if (p.head_dim <= 64) {
    hipLaunchKernelGGL(attn_f32_kernel<64>, grid, block, 0, s, p);
  } else if (p.head_dim <= 128) {
    hipLaunchKernelGGL(attn_f32_kernel<128>, grid, block, 0, s, p);
  } else {
    return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ---------------------------------------------------------------------------
// Rotary embedding of the q and k columns of an fp32 qkv buffer, in place: one
// thread per (row, q|k, head, pair j < head_dim / 2); pair (j, j + head_dim/2)
// of the head turns by 2 pi * frac(pos[r] * freq[j]).
__global__ __launch_bounds__(256) void rope_f32_kernel(float* qkv, int d, int head_dim, const int* m_ptr,
                                                       int m_ub, const int* pos, const double* freq) {
  const int M = rows_from(m_ptr, m_ub);
  const int half = head_dim >> 1;
  const int per_row = d;                 // 2 d columns rotated in pairs: d pairs per row
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const int row = (int)(t / per_row);
  if (row >= M) return;
  const int k = (int)(t % per_row);      // pair index over q and k
  const int head = k / half, j = k % half;
  float* x = qkv + (size_t)row * 3 * d + head * head_dim + j;
  double rv = (double)pos[row] * freq[j];
  rv -= floor(rv);
  const float a = (float)rv;
  const float sn = __builtin_amdgcn_sinf(a), cs = __builtin_amdgcn_cosf(a);
  const float x1 = x[0], x2 = x[half];
  x[0] = x1 * cs - x2 * sn;
  x[half] = x2 * cs + x1 * sn;
}

int launch_rope_f32(float* qkv, int d, int n_heads, int head_dim, const int* m_ptr, int m_ub,
                    const int* pos, const double* freq, hipStream_t s) {
  (void)n_heads;
  if (head_dim % 2 != 0) return -1;
  const long long work = (long long)m_ub * d;
  dim3 grid((unsigned)((work + 255) / 256)), block(256);
  hipLaunchKernelGGL(rope_f32_kernel, grid, block, 0, s, qkv, d, head_dim, m_ptr, m_ub, pos, freq);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace seer
