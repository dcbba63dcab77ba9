// Variable-length bidirectional attention on gfx950 matrix cores (bf16, head_dim 128).
//
// Every query of a sequence attends to every key of the same sequence -- no
// causal mask (the denoising step sees the whole window, Sec. 3.1; logits
// q.k / sqrt(head_dim) and a softmax over the sequence, Sec. 3.6).  Keys at
// positions >= seqused[b] are masked and those query rows get a zero output
// (the static-bucket padding of Sec. 3.5).  With a prefix cache (KV-cache
// compatibility, Appendix D) the keys are the cached prefix rows followed by
// the sequence's own rows.
//
// Design: one workgroup = (sequence, 128-query tile, head); four waves of 32
// queries.  K and V tiles of 64 keys are staged in LDS, double-buffered, and
// shared by the four waves.  Scores are computed transposed, S^T = K Q^T (32x32x16 bf16 MFMA), so
// that each lane owns one query column: the online-softmax statistics are
// per-lane values and the probabilities already sit in the B-operand layout
// of the next product O^T = V^T P^T -- no shuffle of P through LDS.  V arrives
// in fp16 (the QKV projection stores it so) and is staged row-major like K;
// its A-operand fragments (8 keys of one dim per lane) come from pairs of LDS
// transpose reads (ds_read_b64_tr_b16).  The P V product runs in
// fp16: the probabilities keep three more mantissa bits than bf16 would give.
// The softmax's reference maximum is set on a sequence's first key tile and
// moved only when a later tile overflows the fp16 probabilities: the common
// tile takes no maximum at all, and the O rescale is rare.
#include <math.h>

#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace seer {

namespace {

constexpr int QT = 128;   // queries per workgroup
constexpr int KT = 64;    // keys per LDS tile
constexpr int DH = 128;   // head dim
constexpr int NT = 256;
constexpr int K_ROW = DH * 2;   // 256 bytes per key row of K and of V

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef short v8i16_t __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;

}  // namespace

__global__ __launch_bounds__(NT, 2) void attn_bf16_kernel(AttnParams p) {
  // two K/V buffers: tile t+1 is written into one while tile t is read from the other
  // two K/V buffers, each its own array so that the compiler sees reads of one
  // as independent of the direct-to-LDS loads filling the other
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds0[KT * K_ROW];
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds1[KT * K_ROW];
  __shared__ __attribute__((aligned(1024))) uint8_t v_lds0[KT * K_ROW];
  __shared__ __attribute__((aligned(1024))) uint8_t v_lds1[KT * K_ROW];

  // ---- which (sequence, query tile, head) this block owns -------------------
  // Units are (head, query tile over the batch), query tiles fastest; each XCD
  // takes a contiguous range of them, so the query tiles of one sequence and
  // head run together on one XCD and find their K and V tiles in its L2.
  int xt, h;
  {
    const int gx = gridDim.x;
    const int w = xcd_remap(blockIdx.x + gx * blockIdx.y, gx * gridDim.y);
    xt = w % gx;
    h = w / gx;
  }
  int b = -1, t = 0;
  {
    int acc = 0;
    const int j = xt;
    for (int s = 0; s < p.B; ++s) {
      int len = p.cu[s + 1] - p.cu[s];
      len = len < 0 ? 0 : len;
      const int nt = (len + QT - 1) / QT;
      if (j < acc + nt) { b = s; t = j - acc; break; }
      acc += nt;
    }
  }
  if (b < 0) return;
  const int s0 = p.cu[b];
  if (s0 < 0 || s0 >= p.rows_ub) return;
  int len = p.cu[b + 1] - s0;
  len = len > p.rows_ub - s0 ? p.rows_ub - s0 : len;   // never touch rows past the bound
  if (t * QT >= len) return;
  int used = p.used ? p.used[b] : len;
  used = used < 0 ? 0 : (used > len ? len : used);
  // keys: the cached prefix rows (if any), then the sequence's own used rows
  int P = 0, kv0 = 0;
  if (p.cu_kv) {
    kv0 = p.cu_kv[b];
    P = p.cu_kv[b + 1] - kv0;
    P = P < 0 ? 0 : P;
  }
  // Key positions: cache rows at [0, P), own rows at [P4, P4 + used) with P4 =
  // P rounded up to a multiple of 4, so that the 4 rows of one staging load
  // come from one source; the (at most 3) positions [P, P4) are masked.
  const int P4 = (P + 3) & ~3;
  const int nk = used > 0 ? P4 + used : P;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int fr = lane & 31;
  const int fhalf = lane >> 5;
  const uint32_t ld = 3u * (uint32_t)p.d;
  // rows of this sequence; every offset below is < rows_ub * 3 d (checked on the host)
  const uint16_t* seq = static_cast<const uint16_t*>(p.qkv) + (size_t)s0 * ld;
  uint16_t* out = static_cast<uint16_t*>(p.out);

  const int q_row = t * QT + wave * 32 + fr;            // query row inside the sequence
  const int q_src = q_row < len ? q_row : len - 1;

  // Q as the B operand of S^T = K Q^T: lane holds query fr, dims 16*ks + 8*fhalf .. +8.
  bf16x8_t qf[8];
  {
    const uint16_t* qp = seq + (uint32_t)q_src * ld + h * DH + fhalf * 8;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) qf[ks] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4_t*>(qp + ks * 16));
  }

  f32x16_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[i][r] = 0.0f;
  float m_run = -INFINITY;
  float l_run = 0.0f;
  const float c = p.scale * 1.4426950408889634f;

  // ---- K/V tile staging -------------------------------------------------------
  // Direct-to-LDS buffer loads: one load moves 64 x 16 bytes into 1 KiB of
  // consecutive LDS, i.e. 4 key rows of 256 bytes.  Load q of wave w fills tile
  // rows 16 w + 4 q + lane/16 at LDS position lane%16, so the lane fetches the
  // 16-byte dim chunk that the swizzle puts there: (lane%16) ^ (row%16) for K,
  // (lane%16) ^ 4 (row%4) for V (V fragments are read with the LDS transpose
  // read, whose 8-byte accesses then hit distinct banks).  The 4 positions of
  // one load are all cache rows (below P4) or all own rows, so the descriptor
  // and row stride are chosen per wave; gap positions re-read cache row P-1,
  // positions at or past nk re-read the last key (all masked below).
  // Offsets are bytes from the sequence's first qkv row and the sequence's
  // first cache row (< 4 GiB, checked by the host).
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const __amdgpu_buffer_rsrc_t rs_q = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(seq), 0, -1, 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_c = __builtin_amdgcn_make_buffer_rsrc(
      p.cu_kv ? const_cast<uint16_t*>(static_cast<const uint16_t*>(p.kv) + (size_t)kv0 * 2 * p.d)
              : const_cast<uint16_t*>(seq), 0, -1, 0x00020000);
  const uint32_t q_row_bytes = 3u * (uint32_t)p.d * 2u, c_row_bytes = 4u * (uint32_t)p.d;
  const uint32_t k_col = (uint32_t)(p.d + h * DH) * 2u, c_col = (uint32_t)(h * DH) * 2u, v_step = (uint32_t)p.d * 2u;
  auto dma_tile = [&](int kbase, auto buf_tag) {
    constexpr int B_ = decltype(buf_tag)::value;
    uint8_t* kb = B_ ? k_lds1 : k_lds0;
    uint8_t* vb = B_ ? v_lds1 : v_lds0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = 16 * wv + 4 * q + (lane >> 4);
      int key = kbase + r;
      key = key < nk ? key : nk - 1;
      const uint32_t ck = (uint32_t)(((lane & 15) ^ (r & 15)) << 4);
      const uint32_t cv = (uint32_t)(((lane & 15) ^ (4 * (r & 3))) << 4);
      lds_void_t* kd = (lds_void_t*)(kb + (16 * wv + 4 * q) * K_ROW);
      lds_void_t* vd = (lds_void_t*)(vb + (16 * wv + 4 * q) * K_ROW);
      const bool cache = kbase + 16 * wv + 4 * q < P4 || used == 0;
      const int row = cache ? (key < P ? key : P - 1) : key - P4;
      const uint32_t ro = (uint32_t)row * (cache ? c_row_bytes : q_row_bytes) + (cache ? c_col : k_col);
      const __amdgpu_buffer_rsrc_t rs = cache ? rs_c : rs_q;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, kd, 16, ro + ck, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, vd, 16, ro + v_step + cv, 0, 0, 0);
    }
  };

  const int n_kv = (nk + KT - 1) / KT;
  if (n_kv > 0) dma_tile(0, std::integral_constant<int, 0>{});
  // Drain every global load issued so far (Q and tile 0) before the loop.  The
  // wait-count insertion merges the loop entry with the back edge; with Q
  // possibly in flight at entry it would make the first score MFMAs of every
  // iteration wait for the next tile's loads.
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0x0f70);       // vmcnt(0), other counters unconstrained
  __builtin_amdgcn_sched_barrier(0);
  __syncthreads();
  // One tile: scores, online softmax, P V.  BUF is the LDS buffer holding the
  // tile (compile-time, so every fragment address is a loop-invariant base
  // plus an immediate); the next tile goes to the other buffer.
  auto tile_step = [&](int kt, auto buf_tag) {
    constexpr int BUF = decltype(buf_tag)::value;
    const int kbase = kt * KT;
    const uint8_t* kl = BUF ? k_lds1 : k_lds0;
    const uint8_t* vl = BUF ? v_lds1 : v_lds0;
    if (kt + 1 < n_kv) dma_tile(kbase + KT, std::integral_constant<int, BUF ^ 1>{});

    // S^T for 64 keys: two 32-key MFMA row tiles, walked over the 8 dim
    // slices with the next slice's two K fragments read one step ahead.
    f32x16_t s[2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[i][r] = 0.0f;
    {
      const uint8_t* krow = kl + fr * K_ROW;        // keys fr and 32 + fr
      auto kread = [&](int ks, bf16x8_t* dst) {
        const int ch = (2 * ks + fhalf) ^ (fr & 15);
#pragma unroll
        for (int i = 0; i < 2; ++i)
          dst[i] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4_t*>(krow + i * 32 * K_ROW + ch * 16));
      };
      bf16x8_t kf[2][2];
      __builtin_amdgcn_sched_barrier(0);
      kread(0, kf[0]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        if (ks + 1 < 8) kread(ks + 1, kf[(ks + 1) & 1]);
#pragma unroll
        for (int i = 0; i < 2; ++i)
          s[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks & 1][i], qf[ks], s[i], 0, 0, 0);
        if (ks + 1 < 8) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // positions at or past nk only occur in the last tile, gap positions in
    // the tile holding P
    if (kbase + KT > nk || (P < P4 && kbase < P4 && kbase + KT > P)) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kbase + i * 32 + (r >> 2) * 8 + fhalf * 4 + (r & 3);
          if (key >= nk || (key >= P && key < P4)) s[i][r] = -INFINITY;
        }
    }
    // Probabilities against the reference maximum, packed to fp16 as the
    // P V product takes them, and their row sum over the packed values (one
    // v_dot2_f32_f16 with (1, 1) per pair, accumulated in fp32).
    f16x8_t pf[4];
    float lsum;
    auto probs = [&]() {
      const float mc = m_run * c;
      const f16x2_t one2 = {(_Float16)1.0f, (_Float16)1.0f};
      lsum = 0.0f;
#pragma unroll
      for (int sl = 0; sl < 4; ++sl) {
        const int i = sl >> 1, hf = sl & 1;
        u32x4_t pk;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = __builtin_amdgcn_exp2f(s[i][hf * 8 + 2 * e] * c - mc);
          const float p1 = __builtin_amdgcn_exp2f(s[i][hf * 8 + 2 * e + 1] * c - mc);
          const f16x2_t h = __builtin_convertvector(f32x2_t{p0, p1}, f16x2_t);
          lsum = __builtin_amdgcn_fdot2(h, one2, lsum, false);
          pk[e] = __builtin_bit_cast(uint32_t, h);
        }
        pf[sl] = __builtin_bit_cast(f16x8_t, pk);
      }
    };
    // The reference maximum is set on the first tile and moved only when a
    // later tile holds a probability fp16 cannot represent (a score about 16
    // log2 units above it): its row sum is then inf, and the tile is redone
    // against the true running maximum, with O and the sum rescaled.  Any
    // reference at or below the running maximum gives the same softmax; the
    // common tile skips the maximum.
    bool redo = kt == 0;
    if (!redo) {
      probs();
      redo = __any(!(lsum < INFINITY));
    }
    if (redo) {
      float mt = s[0][0];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[i][r]);
      // lanes l and l ^ 32 each hold 32 of the tile's 64 keys of one query's
      // column (alternate groups of four): a register swap across the pair,
      // no LDS round trip
      const u32x2_t sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mt), __float_as_uint(mt), false, false);
      mt = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
      const float m_new = fmaxf(m_run, mt);
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[i][r] *= alpha;
      probs();
    }
    l_run += lsum;

    // O^T += V^T P^T over four 16-key slices x four 32-dim tiles; the V^T
    // fragment of step n + 2 is read while step n multiplies.
    {
      // A operand of step n (16-key slice sl = n/4, 32-dim tile dt = n%4): lane
      // l needs 8 keys of dim 32 dt + l%32, in the order the P fragment holds
      // them (keys 16 hf + 4 kh + 0..3, then + 8).  In each group of 16 lanes
      // the transpose read hands lane j element j%4 of lanes 4e + j/4, e < 4;
      // so lane i of the group points at key K0 + i/4, dims C + 4 (i%4) .. +3,
      // and lane j receives keys K0 .. K0+3 of dim C + j.
      const int il = lane & 15;
      const int vkey = 4 * (lane >> 5) + (il >> 2);           // + 32 i + 16 hf (+ 8)
      const int vc8 = 4 * ((lane >> 4) & 1) + (il & 3);        // + 8 dt, 8-byte chunk
      const uint8_t* vrow = vl + vkey * K_ROW;
      auto vread = [&](int n) {
        const int sl = n >> 2, dt = n & 3;
        const int key0 = 32 * (sl >> 1) + 16 * (sl & 1);
        const int c8 = (8 * dt + vc8) ^ (8 * (vkey & 3));
        const uint8_t* a = vrow + key0 * K_ROW + (c8 << 3);
        const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)a);
        const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(a + 8 * K_ROW));
        return __builtin_bit_cast(f16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      };
      f16x8_t vf[3];
      __builtin_amdgcn_sched_barrier(0);
      vf[0] = vread(0);
      vf[1] = vread(1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int n = 0; n < 16; ++n) {
        if (n + 2 < 16) vf[(n + 2) % 3] = vread(n + 2);
        o[n & 3] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf[n % 3], pf[n >> 2], o[n & 3], 0, 0, 0);
        if (n + 2 < 16) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // Buffer BUF^1 was last read in tile kt-1, which every wave left through
    // the barrier below; this wave's loads of tile kt+1 have landed once
    // vmcnt is zero, and one barrier then publishes the whole tile.
    __builtin_amdgcn_s_waitcnt(0x0f70);
    __syncthreads();
  };
  for (int kt = 0; kt < n_kv; kt += 2) {
    tile_step(kt, std::integral_constant<int, 0>{});
    if (kt + 1 < n_kv) tile_step(kt + 1, std::integral_constant<int, 1>{});
  }

  // ---- normalise and store ----------------------------------------------------
  const float l_tot = l_run + __shfl_xor(l_run, 32, kWave);
  if (q_row < len) {
    const bool real = q_row < used;
    const float inv = (real && l_tot > 0.0f) ? 1.0f / l_tot : 0.0f;
    uint16_t* op = out + (size_t)(s0 + q_row) * p.d + h * DH + fhalf * 4;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 v;
        v.x = pack_bf2(o[dt][g * 4 + 0] * inv, o[dt][g * 4 + 1] * inv);
        v.y = pack_bf2(o[dt][g * 4 + 2] * inv, o[dt][g * 4 + 3] * inv);
        *reinterpret_cast<uint2*>(op + dt * 32 + g * 8) = v;
      }
  }
}

int launch_attn_bf16(const AttnParams& p, hipStream_t s) {
  if (p.head_dim != DH) return -1;
  // byte offsets inside the qkv rows and the cache rows are 32-bit
  if ((uint64_t)p.rows_ub * 3u * (uint64_t)p.d * 2u >= (1ull << 32)) return -1;
  if (p.cu_kv && !p.kv) return -1;
  dim3 grid((p.rows_ub + QT - 1) / QT + p.B, p.n_heads), block(NT);
  hipLaunchKernelGGL(attn_bf16_kernel, grid, block, 0, s, p);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace seer
