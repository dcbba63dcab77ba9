// Row statistics, the SNR boundary scan, routing + compaction and weight prepack.
#include "common.h"
#include "kernels.h"

namespace seer {

// ---------------------------------------------------------------------------
// inv_rms[r] = 1/sqrt(mean(x[r]^2) + eps): one wave per row, fixed reduction
// order (deterministic).  The RMSNorm itself is folded into the following
// GEMM: (x * inv_rms) W^T = inv_rms * (x W^T).
template <bool BF16>
__global__ __launch_bounds__(256) void rms_inv_kernel(const void* x, int ld, int d, const int* m_ptr,
                                                      int m_ub, float eps, float* out, RopeArgs rope) {
  const int M = rows_from(m_ptr, m_ub);
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (rope.pos && blockIdx.x == 0 && threadIdx.x < rope.head_dim / 2) {
    const int j = threadIdx.x;
    rope.freq[j] = pow((double)rope.theta, -2.0 * j / rope.head_dim) / 6.283185307179586;   // / (2 pi)
  }
  if (row >= M) return;
  if (rope.pos && lane == 0) {
    // sequence of the row: the last b with cu[b] <= row
    int lo = 0, hi = rope.B - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (rope.cu[mid] <= row) lo = mid;
      else hi = mid - 1;
    }
    const int pre = rope.cu_kv ? rope.cu_kv[lo + 1] - rope.cu_kv[lo] : 0;
    rope.pos[row] = row - rope.cu[lo] + (pre > 0 ? pre : 0);
  }
  float acc = 0.0f;
  if constexpr (BF16) {
    const uint16_t* xr = static_cast<const uint16_t*>(x) + (size_t)row * ld;
    auto add = [&](const uint4 v) {
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float lo = __uint_as_float(w[e] << 16);
        const float hi = __uint_as_float(w[e] & 0xffff0000u);
        acc = fmaf(lo, lo, acc);
        acc = fmaf(hi, hi, acc);
      }
    };
    // lane l sums chunks j = 8 l + 512 u in increasing u.  Eight chunks (a
    // whole 4096-wide row) are requested before the first is used, so a row
    // costs one memory latency, not eight; the summation order is unchanged.
    int j = lane * 8;
    for (; j + 512 * 7 < d; j += 512 * 8) {
      uint4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = *reinterpret_cast<const uint4*>(xr + j + 512 * u);
#pragma unroll
      for (int u = 0; u < 8; ++u) add(v[u]);
    }
    for (; j < d; j += 512) add(*reinterpret_cast<const uint4*>(xr + j));
  } else {
    const float* xr = static_cast<const float*>(x) + (size_t)row * ld;
    for (int j = lane; j < d; j += 64) acc = fmaf(xr[j], xr[j], acc);
  }
  acc = wave_sum(acc);
  if (lane == 0) out[row] = 1.0f / sqrtf(acc / (float)d + eps);
}

int launch_rms_inv(bool bf16, const void* x, int ld, int d, const int* m_ptr, int m_ub, float eps,
                   float* out, hipStream_t s, const RopeArgs* rope) {
  dim3 grid((m_ub + 3) / 4), block(256);
  RopeArgs r{};
  if (rope) r = *rope;
  if (bf16)
    hipLaunchKernelGGL(rms_inv_kernel<true>, grid, block, 0, s, x, ld, d, m_ptr, m_ub, eps, out, r);
  else
    hipLaunchKernelGGL(rms_inv_kernel<false>, grid, block, 0, s, x, ld, d, m_ptr, m_ub, eps, out, r);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

__global__ void zero_i32_kernel(int* p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

int launch_zero_i32(int* p, int n, hipStream_t s) {
  if (n <= 0) return 0;
  int blocks = (n + 255) / 256;
  blocks = blocks > 1024 ? 1024 : blocks;
  hipLaunchKernelGGL(zero_i32_kernel, dim3(blocks), dim3(256), 0, s, p, n);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ---------------------------------------------------------------------------
// SNR jump/plateau scan (Sec. 3.3), one workgroup per sequence.  Each thread
// tests candidate positions i = 1 + tid, 1 + tid + 256, ... in increasing
// order and stops at its first hit; the block minimum is the leftmost hit.
// With s_i = c_i / I the two conditions are compared in exact 64-bit integers:
//   jump  >= tau        <=>  tau_den * (min W - c_{i-1}) >= tau_num * I
//   noise <= gamma*jump <=>  gamma_den * (max W - min W) <= gamma_num * (min W - c_{i-1})
__global__ __launch_bounds__(256) void detect_kernel(DetectParams p) {
  __shared__ int s_min[4];
  const int b = blockIdx.x;
  const int base = p.cu[b] + p.win_off[b];
  // the window never reaches past its own sequence
  int n = p.win_len[b];
  const int room = p.cu[b + 1] - base;
  n = n > room ? room : n;
  n = n < 0 ? 0 : n;
  const int w = p.lookahead;
  const int* c = p.cnt + base;
  int best = n;
  for (int i = 1 + (int)threadIdx.x; i + w <= n; i += 256) {
    int mn = c[i], mx = c[i];
    for (int t = 1; t < w; ++t) {
      const int v = c[i + t];
      mn = v < mn ? v : mn;
      mx = v > mx ? v : mx;
    }
    const long long dj = (long long)mn - (long long)c[i - 1];
    const long long dn = (long long)mx - (long long)mn;
    if ((long long)p.tau_den * dj >= (long long)p.tau_num * (long long)p.d_ff &&
        (long long)p.gamma_den * dn <= (long long)p.gamma_num * dj) {
      best = i;
      break;
    }
  }
  best = wave_min_int(best);
  if ((threadIdx.x & 63) == 0) s_min[threadIdx.x >> 6] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    int m = s_min[0];
    for (int k = 1; k < 4; ++k) m = s_min[k] < m ? s_min[k] : m;
    p.boundary[b] = m;
    p.keep_len[b] = m < n ? m + 1 : n;
  }
}

int launch_detect(const DetectParams& p, hipStream_t s) {
  hipLaunchKernelGGL(detect_kernel, dim3(p.B), dim3(256), 0, s, p);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ---------------------------------------------------------------------------
// Kept row tiles after the scan (the rows the compaction copies), so that the
// detection layer's down projection computes only those.  Thread t of each
// 1024-tile chunk finds the first sequence reaching into tile t by bisection
// of cu and walks the sequences that start inside it; the live tiles are
// then listed in order (wave ballots, per-wave counts in LDS).
__global__ __launch_bounds__(1024) void kept_tiles_kernel(KeptTilesParams p) {
  __shared__ int s_wave[16];
  __shared__ int s_base;
  const int M = rows_from(p.cu + p.B, p.rows_ub);
  const int tiles = (M + 255) / 256;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (threadIdx.x == 0) s_base = 0;
  __syncthreads();
  for (int t0 = 0; t0 < tiles; t0 += 1024) {
    const int t = t0 + (int)threadIdx.x;
    bool live = false;
    if (t < tiles) {
      const int r0 = 256 * t, r1 = min(r0 + 256, M);
      int lo = 0, hi = p.B - 1;               // last b with cu[b] <= r0
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (p.cu[mid] <= r0) lo = mid; else hi = mid - 1;
      }
      for (int b = lo; b < p.B && !live; ++b) {
        const int s0 = p.cu[b];
        if (s0 >= r1) break;
        const int len = p.cu[b + 1] - s0;
        int keep = p.keep_len[b];
        keep = keep < 0 ? 0 : (keep > p.win_len[b] ? p.win_len[b] : keep);
        int used = p.win_off[b] + keep;
        used = used < 0 ? 0 : (used > len ? len : used);
        live = max(s0, r0) < min(s0 + used, r1);
      }
    }
    const unsigned long long bal = __ballot(live);
    const int below = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) s_wave[wv] = __popcll(bal);
    __syncthreads();
    int off = s_base;
    for (int k = 0; k < wv; ++k) off += s_wave[k];
    if (live) p.map[1 + off + below] = t;
    __syncthreads();
    if (threadIdx.x == 0) {
      int n = 0;
      for (int k = 0; k < 16; ++k) n += s_wave[k];
      s_base += n;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) p.map[0] = s_base;
}

int launch_kept_tiles(const KeptTilesParams& p, hipStream_t s) {
  hipLaunchKernelGGL(kept_tiles_kernel, dim3(1), dim3(1024), 0, s, p);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ---------------------------------------------------------------------------
// Routing + compaction (Sec. 3.4-3.5).  Every workgroup rebuilds the routing
// plan of the (small) batch in LDS -- classes, buckets, padding waste, paths,
// allocations and the exclusive prefix sum of the packed lengths -- so a
// single launch both routes and moves the rows, with no host round trip.
// Workgroup 0 publishes cu_dst, seqused, route and the control word.
namespace {
constexpr int kRows = 8;       // destination rows per workgroup
constexpr int kMaxClass = 32;

__device__ __forceinline__ int coarse_class(int L) {
  const int m = L > 8 ? L : 8;
  int k = 0;
  long long p4 = 1;
  while (p4 < m) { p4 *= 4; ++k; }
  return k;
}

// keep_len clamped to [0, win_len]
__device__ __forceinline__ int clamp_keep(const RepackParams& p, int b) {
  const int k = p.keep_len[b];
  const int n = p.win_len[b];
  return k < 0 ? 0 : (k > n ? n : k);
}

__device__ __forceinline__ int bucket_of(int L, int nmax) {
  int bk = 8;
  while (bk < nmax) {
    if (bk >= L) return bk;
    bk <<= 1;
  }
  return nmax;
}
}  // namespace

__global__ __launch_bounds__(256) void repack_kernel(RepackParams p) {
  __shared__ int s_cu[kRepackMaxBatch + 1];
  __shared__ int s_used[kRepackMaxBatch];
  __shared__ int s_src[kRepackMaxBatch];
  __shared__ int s_alloc[kRepackMaxBatch];
  __shared__ int s_part[256];
  __shared__ unsigned long long c_sum[kMaxClass];
  __shared__ int c_cnt[kMaxClass], c_max[kMaxClass], c_path[kMaxClass], c_bucket[kMaxClass],
      c_gid[kMaxClass];
  __shared__ int s_nmax, s_kmax, s_total, s_cap, s_status, s_ngroups;

  const int tid = threadIdx.x;
  const int B = p.B;
  if (tid < kMaxClass) { c_sum[tid] = 0; c_cnt[tid] = 0; c_max[tid] = 0; }
  if (tid == 0) { s_nmax = 0; s_kmax = 0; }
  __syncthreads();
  for (int b = tid; b < B; b += 256) {
    const int keep = clamp_keep(p, b);
    // rows of sequence b that are copied: its prefix and kept window, or with
    // window_only the kept window alone
    const int pre = p.window_only ? 0 : p.win_off[b];
    const int skip = p.window_only ? p.win_off[b] : 0;
    int used = pre + keep;
    const int len = p.cu_src[b + 1] - p.cu_src[b] - skip;
    s_used[b] = used < len ? (used > 0 ? used : 0) : (len > 0 ? len : 0);   // copies stay inside the source sequence
    s_src[b] = p.cu_src[b] + skip;
    atomicMax(&s_nmax, p.win_len[b]);
    atomicMax(&s_kmax, keep);
    const int k = coarse_class(keep);
    atomicAdd(&c_cnt[k], 1);
    atomicAdd(&c_sum[k], (unsigned long long)keep);
    atomicMax(&c_max[k], keep);
  }
  __syncthreads();
  if (tid < kMaxClass) {
    const int k = tid;
    const int n = c_cnt[k];
    int gid = 0;
    for (int j = 0; j < k; ++j) gid += c_cnt[j] > 0 ? 1 : 0;
    c_gid[k] = gid;
    if (n > 0) {
      const int bg = bucket_of(c_max[k], s_nmax);
      c_bucket[k] = bg;
      const long long cap = (long long)n * bg;
      const long long waste = cap - (long long)c_sum[k];
      int path;
      if (n == 1 || c_max[k] <= 4) path = 2;
      else if ((long long)p.tau_den * waste <= (long long)p.tau_num * cap) path = 0;
      else path = 1;
      c_path[k] = path;
    }
  }
  __syncthreads();
  const int naive_bucket = bucket_of(s_kmax, s_nmax);
  for (int b = tid; b < B; b += 256) {
    const int keep = clamp_keep(p, b);
    int alloc;
    if (p.policy == 1) alloc = naive_bucket;
    else if (p.policy == 2) alloc = keep;
    else {
      const int k = coarse_class(keep);
      alloc = c_path[k] == 0 ? c_bucket[k] : keep;
    }
    s_alloc[b] = alloc;
  }
  __syncthreads();
  // exclusive prefix sum of (prefix rows + alloc): 4 consecutive entries per thread
  {
    int local = 0;
    for (int e = 0; e < 4; ++e) {
      const int b = tid * 4 + e;
      if (b < B) local += (p.window_only ? 0 : p.win_off[b]) + s_alloc[b];
    }
    s_part[tid] = local;
    __syncthreads();
    if (tid == 0) {
      int run = 0;
      for (int k = 0; k < 256; ++k) { const int v = s_part[k]; s_part[k] = run; run += v; }
      s_total = run;
      const int g = p.granule > 0 ? p.granule : 1;
      s_cap = (int)(((long long)run + g - 1) / g * g);
      s_status = s_cap > p.dst_capacity_rows ? -3 : 0;
      int ng = 0;
      for (int k = 0; k < kMaxClass; ++k) ng += c_cnt[k] > 0 ? 1 : 0;
      s_ngroups = (p.policy == 0) ? ng : 1;
    }
    __syncthreads();
    int run = s_part[tid];
    for (int e = 0; e < 4; ++e) {
      const int b = tid * 4 + e;
      if (b < B) { s_cu[b] = run; run += (p.window_only ? 0 : p.win_off[b]) + s_alloc[b]; }
    }
    if (tid == 0) s_cu[B] = s_total;
    __syncthreads();
  }
  const bool ok = s_status == 0;

  if (blockIdx.x == 0) {
    for (int b = tid; b <= B; b += 256) p.cu_dst[b] = ok ? s_cu[b] : 0;
    for (int b = tid; b < B; b += 256) {
      const int keep = clamp_keep(p, b);
      int path, gid;
      if (p.policy == 1) { path = 0; gid = 0; }
      else if (p.policy == 2) { path = 1; gid = 0; }
      else { const int k = coarse_class(keep); path = c_path[k]; gid = c_gid[k]; }
      p.seqused[b] = ok ? s_used[b] : 0;
      p.route[3 * b + 0] = path;
      p.route[3 * b + 1] = gid;
      p.route[3 * b + 2] = s_alloc[b];
    }
    if (tid == 0) {
      int ns = 0, nv = 0, ne = 0, mx = 0;
      for (int b = 0; b < B; ++b) {
        int path;
        if (p.policy == 1) path = 0;
        else if (p.policy == 2) path = 1;
        else path = c_path[coarse_class(clamp_keep(p, b))];
        ns += path == 0; nv += path == 1; ne += path == 2;
        mx = s_alloc[b] > mx ? s_alloc[b] : mx;
      }
      int ctrl[9] = {ok ? s_total : 0, ok ? s_cap : 0, ns, nv, ne, s_ngroups, mx, s_status, 1};
      for (int dst = 0; dst < 2; ++dst) {
        int* c = dst == 0 ? p.ctrl_dev : p.ctrl_host;
        if (c == nullptr) continue;
        for (int k = 0; k < 8; ++k) c[k] = ctrl[k];
        __threadfence_system();
        c[8] = ctrl[8];
        __threadfence_system();
      }
    }
  }
  if (!ok) return;

  const int nchunk = p.row_bytes >> 4;
  const int r0 = blockIdx.x * kRows;
  for (int rr = 0; rr < kRows; ++rr) {
    const int r = r0 + rr;
    if (r >= s_cap) break;
    int src_row = -1;
    if (r < s_total) {
      int lo = 0, hi = B - 1;      // last b with s_cu[b] <= r
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s_cu[mid] <= r) lo = mid; else hi = mid - 1;
      }
      const int local = r - s_cu[lo];
      if (local < s_used[lo]) src_row = s_src[lo] + local;
    }
    for (int bi = 0; bi < p.n_buffers; ++bi) {
      uint4* d = reinterpret_cast<uint4*>(p.dst[bi] + (size_t)r * p.row_bytes);
      if (src_row >= 0) {
        const uint4* sp = reinterpret_cast<const uint4*>(p.src[bi] + (size_t)src_row * p.row_bytes);
        for (int c = tid; c < nchunk; c += 256) d[c] = sp[c];
      } else {
        const uint4 z = make_uint4(0, 0, 0, 0);
        for (int c = tid; c < nchunk; c += 256) d[c] = z;
      }
    }
  }
}

// One workgroup per cache row r: its sequence b (last b with cu_kv[b] <= r),
// source row cu[b] + (r - cu_kv[b]) of the layer call, K | V columns
// [d, 3d) moved as 16-byte chunks.  A prefix longer than its sequence, or a
// source row past the qkv region, leaves the cache row untouched.
__global__ __launch_bounds__(256) void kv_export_kernel(KvExportParams p) {
  const int r = blockIdx.x;
  if (r >= p.cu_kv[p.B]) return;
  int lo = 0, hi = p.B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.cu_kv[mid] <= r) lo = mid; else hi = mid - 1;
  }
  const int j = r - p.cu_kv[lo];
  const int s0 = p.cu[lo];
  if (j >= p.cu[lo + 1] - s0) return;
  const int src = s0 + j;
  if (src < 0 || src >= p.rows_ub) return;
  const size_t rb = (size_t)2 * p.d * p.es;
  const uint4* sp = reinterpret_cast<const uint4*>(p.qkv + (size_t)src * 3 * p.d * p.es + (size_t)p.d * p.es);
  uint4* dp = reinterpret_cast<uint4*>(p.dst + (size_t)r * rb);
  for (int c = threadIdx.x; c < (int)(rb >> 4); c += 256) dp[c] = sp[c];
}

int launch_kv_export(const KvExportParams& p, int kv_rows_ub, hipStream_t s) {
  if (kv_rows_ub < 1) return 0;
  hipLaunchKernelGGL(kv_export_kernel, dim3(kv_rows_ub), dim3(256), 0, s, p);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

int launch_repack(const RepackParams& p, hipStream_t s) {
  int blocks = (p.dst_capacity_rows + kRows - 1) / kRows;
  blocks = blocks < 1 ? 1 : blocks;
  hipLaunchKernelGGL(repack_kernel, dim3(blocks), dim3(256), 0, s, p);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ---------------------------------------------------------------------------
// Weight prepack.  bf16: [Wq;Wk;Wv] (3d x d, the q and k rows of each head in
// block order 0, 2, 1, 3: qk_packed_row), Wo, gate/up interleaved in blocks of
// 32 rows (2I x d), Wd, each stored fragment-major (frag_b_index).  fp32:
// [Wq;Wk;Wv], Wo, Wg, Wu, Wd, row-major.  RMSNorm gains multiply the input
// columns of the projections they feed.
PackedLayout packed_layout(int d, int d_ff, bool bf16) {
  const size_t es = bf16 ? 2 : 4;
  auto up = [](size_t n) { return (n + 127) / 128 * 128; };
  PackedLayout L;
  L.qkv = 0;
  L.o = up(L.qkv + (size_t)3 * d * d);
  L.gu = up(L.o + (size_t)d * d);
  L.dn = up(L.gu + (size_t)2 * d_ff * d);
  L.total_bytes = up(L.dn + (size_t)d * d_ff) * es;
  return L;
}

template <bool BF16>
__global__ void prepack_kernel(PrepackParams p, PackedLayout L) {
  using T = typename std::conditional<BF16, uint16_t, float>::type;
  const int d = p.d, I = p.d_ff;
  T* dst = static_cast<T*>(p.dst);
  auto ld = [](const void* src, size_t idx) -> float {
    if constexpr (BF16) return bf2f(static_cast<const uint16_t*>(src)[idx]);
    else return static_cast<const float*>(src)[idx];
  };
  // packed element (r, k) of a [rows, K] block at base
  auto st = [&](size_t base, size_t r, size_t k, size_t K, float v, const void* src, size_t sidx, bool scaled) {
    if constexpr (BF16) {
      dst[base + frag_b_index(r, k, K)] = scaled ? f2bf(v) : static_cast<const uint16_t*>(src)[sidx];
    } else {
      dst[base + r * K + k] = v;
    }
  };
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  const size_t start = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  // q, k, v
  for (size_t e = start; e < (size_t)3 * d * d; e += stride) {
    const size_t r = e / d, k = e % d;
    const size_t wr = (BF16 && r < (size_t)2 * d) ? qk_packed_row(r) : r;
    const void* src = wr < (size_t)d ? p.wq : (wr < (size_t)2 * d ? p.wk : p.wv);
    const size_t sidx = (wr % d) * d + k;
    const float g = p.g1 ? p.g1[k] : 1.0f;
    st(L.qkv, r, k, d, ld(src, sidx) * g, src, sidx, p.g1 != nullptr);
  }
  for (size_t e = start; e < (size_t)d * d; e += stride) st(L.o, e / d, e % d, d, ld(p.wo, e), p.wo, e, false);
  for (size_t e = start; e < (size_t)2 * I * d; e += stride) {
    const size_t r = e / d, k = e % d;
    const void* src;
    size_t sr;
    if constexpr (BF16) {
      const size_t blk = r / 64, half = (r % 64) / 32, within = r % 32;
      src = half ? p.wu : p.wg;
      sr = blk * 32 + within;
    } else {
      src = r < (size_t)I ? p.wg : p.wu;
      sr = r % I;
    }
    const size_t sidx = sr * d + k;
    const float g = p.g2 ? p.g2[k] : 1.0f;
    st(L.gu, r, k, d, ld(src, sidx) * g, src, sidx, p.g2 != nullptr);
  }
  for (size_t e = start; e < (size_t)d * I; e += stride) st(L.dn, e / I, e % I, I, ld(p.wd, e), p.wd, e, false);
}

int launch_prepack(const PrepackParams& p, hipStream_t s) {
  const PackedLayout L = packed_layout(p.d, p.d_ff, p.bf16);
  dim3 grid(2048), block(256);
  if (p.bf16) hipLaunchKernelGGL(prepack_kernel<true>, grid, block, 0, s, p, L);
  else hipLaunchKernelGGL(prepack_kernel<false>, grid, block, 0, s, p, L);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// One 16-byte destination chunk per thread: chunk c is lane c % 64 of block
// c / 64, i.e. 8 consecutive K values of one row, a 16-byte run of the source.
__global__ void pack_frag_kernel(const uint4* src, int N, int K, uint4* dst) {
  const size_t n_chunks = (size_t)N * K / 8;
  const size_t kb = (size_t)K / 16;
  for (size_t c = (size_t)blockIdx.x * blockDim.x + threadIdx.x; c < n_chunks; c += (size_t)gridDim.x * blockDim.x) {
    const size_t blk = c / 64, l = c % 64;
    const size_t n = (blk / kb) * 32 + l % 32;
    const size_t k = (blk % kb) * 16 + (l / 32) * 8;
    dst[c] = src[(n * K + k) / 8];
  }
}

int launch_pack_frag(const void* src, int N, int K, void* dst, hipStream_t s) {
  if (N % 32 != 0 || K % 16 != 0) return -1;
  hipLaunchKernelGGL(pack_frag_kernel, dim3(4096), dim3(256), 0, s, static_cast<const uint4*>(src), N, K,
                     static_cast<uint4*>(dst));
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ---------------------------------------------------------------------------
// LM-head prediction: one wave per row merges the row's 128-column partials
// in column order (a strict > keeps the smallest column among equal maxima).
__global__ __launch_bounds__(256) void argmax_reduce_kernel(const ArgmaxPartial* part, int n_part, const int* m_ptr,
                                                            int m_ub, int* pred, float* conf) {
  const int M = rows_from(m_ptr, m_ub);
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= M) return;
  const ArgmaxPartial* pr = part + (size_t)row * n_part;
  float m = -INFINITY, sum = 0.0f;
  int a = 0x7fffffff;
  for (int k = lane; k < n_part; k += 64) {
    const ArgmaxPartial v = pr[k];
    if (v.max > m) {
      sum = sum * __expf(m - v.max) + v.sum;
      m = v.max;
      a = v.arg;
    } else {
      sum += v.sum * __expf(v.max - m);
    }
  }
  // lanes hold disjoint column sets: merge by (max desc, column asc)
  for (int off = 32; off > 0; off >>= 1) {
    const float m2 = __shfl_xor(m, off, 64);
    const float s2 = __shfl_xor(sum, off, 64);
    const int a2 = __shfl_xor(a, off, 64);
    const float mm = fmaxf(m, m2);
    const float e1 = m == -INFINITY ? 0.0f : __expf(m - mm);
    const float e2 = m2 == -INFINITY ? 0.0f : __expf(m2 - mm);
    const int at = (m2 > m || (m2 == m && a2 < a)) ? a2 : a;
    sum = sum * e1 + s2 * e2;
    m = mm;
    a = at;
  }
  if (lane == 0) {
    pred[row] = a;
    conf[row] = 1.0f / sum;
  }
}

int launch_argmax_reduce(const void* partials, int n_part, const int* m_ptr, int m_ub, int* pred, float* conf,
                         hipStream_t s) {
  dim3 grid((m_ub + 3) / 4), block(256);
  hipLaunchKernelGGL(argmax_reduce_kernel, grid, block, 0, s, static_cast<const ArgmaxPartial*>(partials), n_part,
                     m_ptr, m_ub, pred, conf);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ---------------------------------------------------------------------------
// Remasking step.  Decision: one workgroup of 1024 per sequence stages the
// keys of its positions in LDS (confidence if masked, -1 if committed; a
// softmax probability is > 0), so a masked position's rank -- the number of
// masked positions with a larger (confidence, -position) key -- is a sweep of
// LDS broadcasts; the k = ceil(n / steps_left) of rank < k are committed.
// Keys are unique, so the selection is exact and independent of the thread
// order.  Rows: a second launch writes the next input rows, 64 workgroups per
// sequence.
constexpr int kRemaskThreads = 1024;
constexpr int kRemaskPerThread = 8;    // up to 8192 positions per sequence

__global__ __launch_bounds__(kRemaskThreads) void remask_decide_kernel(RemaskParams p) {
  __shared__ __attribute__((aligned(16))) float s_key[kRemaskThreads * kRemaskPerThread];
  __shared__ int s_cnt;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int r0 = p.cu[b];
  const int rows = p.cu[b + 1] - r0;
  int used = p.used ? p.used[b] : rows;
  used = used < 0 ? 0 : (used > rows ? rows : used);
  used = used > p.max_used ? p.max_used : used;
  if (tid == 0) s_cnt = 0;
  __syncthreads();
  int local = 0;
  for (int i = tid; i < ((used + 7) & ~7); i += kRemaskThreads) {
    const bool masked = i < used && p.tokens[r0 + i] < 0;
    s_key[i] = i < used ? (masked ? p.conf[r0 + i] : -1.0f) : -2.0f;
    local += masked;
  }
  if (local) atomicAdd(&s_cnt, local);
  __syncthreads();
  const int n = s_cnt;
  const int k = p.steps_left <= 1 ? n : (n + p.steps_left - 1) / p.steps_left;
#pragma unroll
  for (int t = 0; t < kRemaskPerThread; ++t) {
    const int i = tid + kRemaskThreads * t;
    if (i >= used || k == 0) continue;
    const float ci = s_key[i];
    if (ci < 0.0f) continue;
    // eight keys per step (two 16-byte LDS reads in flight); keys past `used`
    // are -2 (below every key), so whole steps need no bounds test
    int rank = 0;
    for (int j0 = 0; j0 < used && rank < k; j0 += 8) {
      const f32x4_t c0 = *reinterpret_cast<const f32x4_t*>(&s_key[j0]);
      const f32x4_t c1 = *reinterpret_cast<const f32x4_t*>(&s_key[j0 + 4]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        rank += (c0[e] > ci) || (c0[e] == ci && j0 + e < i);
        rank += (c1[e] > ci) || (c1[e] == ci && j0 + 4 + e < i);
      }
    }
    if (rank < k) {
      int tok = p.pred[r0 + i];
      tok = tok < 0 ? 0 : (tok >= p.vocab ? p.vocab - 1 : tok);
      p.tokens[r0 + i] = tok;        // only this thread reads or writes entry i from here on
    }
  }
}

constexpr int kRemaskRowSplit = 64;

__global__ __launch_bounds__(256) void remask_rows_kernel(RemaskParams p) {
  const int b = blockIdx.x;
  const int r0 = p.cu[b];
  const int rows = p.cu[b + 1] - r0;
  int used = p.used ? p.used[b] : rows;
  used = used < 0 ? 0 : (used > rows ? rows : used);
  used = used > p.max_used ? p.max_used : used;
  const int per = (rows + kRemaskRowSplit - 1) / kRemaskRowSplit;
  const int i0 = blockIdx.y * per;
  const int i1 = i0 + per < rows ? i0 + per : rows;
  const int chunks = p.d >> 3;
  for (int c = threadIdx.x; c < (i1 - i0) * chunks; c += 256) {
    const int i = i0 + c / chunks, ch = c % chunks;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (i < used) {
      const int tok = p.tokens[r0 + i];
      const uint16_t* src = tok >= 0 ? p.emb + (size_t)tok * p.d : p.x0 + (size_t)(r0 + i) * p.d;
      v = reinterpret_cast<const uint4*>(src)[ch];
    }
    reinterpret_cast<uint4*>(p.x_next + (size_t)(r0 + i) * p.d)[ch] = v;
  }
}

int launch_remask(const RemaskParams& p, hipStream_t s) {
  if (p.max_used > kRemaskThreads * kRemaskPerThread || p.d % 8 != 0) return -1;
  hipLaunchKernelGGL(remask_decide_kernel, dim3(p.B), dim3(kRemaskThreads), 0, s, p);
  if (hipGetLastError() != hipSuccess) return -1;
  hipLaunchKernelGGL(remask_rows_kernel, dim3(p.B, kRemaskRowSplit), dim3(256), 0, s, p);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace seer
