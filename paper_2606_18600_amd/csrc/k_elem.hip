// Row-wise and element-wise kernels of a decoder layer: RMSNorm (fused with
// the stage-input conversion, or with the residual add of split-K partial
// sums), per-head q/k RMSNorm + RoPE + paged KV write, SwiGLU, and the
// stage-output cast.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "packed.hpp"

namespace stage_k {

namespace {

// RMSNorm: one block per row; the row is held in registers (16384 / 4 /
// threads float4 per thread), so each kernel is one round trip to memory.
// H is a multiple of 4 and at most 16384.

template <typename T> struct vec4_io;
template <> struct vec4_io<float> {
  __device__ static __forceinline__ float4 load(const float* p, size_t i) {
    return *(const float4*)(p + i);
  }
};
template <> struct vec4_io<bf16_t> {
  __device__ static __forceinline__ float4 load(const bf16_t* p, size_t i) {
    const u32x2_t w = *(const u32x2_t*)(p + i);
    return make_float4(lo_bf16(w[0]), hi_bf16(w[0]), lo_bf16(w[1]), hi_bf16(w[1]));
  }
};

__device__ __forceinline__ void add4(float4& a, const float4 b) {
  a.x += b.x;
  a.y += b.y;
  a.z += b.z;
  a.w += b.w;
}

// Store 4 consecutive columns k..k+3 (k % 4 == 0) of row t of an activation:
// bf16 into the packed layout (8 contiguous bytes), fp32 row-major.
__device__ __forceinline__ void store_act4(bf16_t* h, int t, int k, int K, float4 v) {
  u32x2_t w;
  w[0] = pack_bf16x2(v.x, v.y);
  w[1] = pack_bf16x2(v.z, v.w);
  *(u32x2_t*)(h + packed_a_offset(t, k, K)) = w;
}
__device__ __forceinline__ void store_act4(float* h, int t, int k, int K, float4 v) {
  *(float4*)(h + (size_t)t * K + k) = v;
}

// kS: number of split-K partial planes added to x (compile time, so that all
// of a thread's loads are issued together); rows before r0 have none. With
// kEmbed, row t reads input row rows[t] (rows == nullptr: row t).
template <typename InT, typename OutT, bool kEmbed, int kThreads, int kS>
__global__ __launch_bounds__(kThreads) void rmsnorm_kernel(const InT* __restrict__ in,
                                                           const int32_t* __restrict__ rows,
                                                           float* __restrict__ x,
                                                           const float* __restrict__ part, int T,
                                                           int r0, OutT* __restrict__ h,
                                                           const OutT* __restrict__ gain, int H,
                                                           float eps) {
  constexpr int kVec = 16384 / 4 / kThreads;
  const int t = blockIdx.x;
  const size_t row = (size_t)t * H;
  const size_t in_row = kEmbed && rows != nullptr ? (size_t)rows[t] * H : row;
  const size_t plane = (size_t)(T - r0) * H;
  const size_t prow = (size_t)(t - r0) * H;  // this row in the partial planes (t >= r0)
  const bool adds = kS > 0 && t >= r0;
  const int H4 = H >> 2;
  __shared__ float red[kThreads / STAGE_WAVE];
  float4 v[kVec];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kVec; ++j) {
    const int i4 = threadIdx.x + j * kThreads;
    if (i4 < H4) {
      const size_t e = row + 4 * (size_t)i4;
      if constexpr (kEmbed)
        v[j] = vec4_io<InT>::load(in, in_row + 4 * (size_t)i4);
      else
        v[j] = *(const float4*)(x + e);
      if (adds) {
        float4 p[kS > 0 ? kS : 1];
#pragma unroll
        for (int sp = 0; sp < kS; ++sp)
          p[sp] = *(const float4*)(part + sp * plane + prow + 4 * (size_t)i4);
#pragma unroll
        for (int sp = 0; sp < kS; ++sp) add4(v[j], p[sp]);
      }
      if (kEmbed || adds) *(float4*)(x + e) = v[j];
      ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
    }
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kThreads / STAGE_WAVE; ++w) tot += red[w];
  const float r = 1.0f / sqrtf(tot / (float)H + eps);
#pragma unroll
  for (int j = 0; j < kVec; ++j) {
    const int i4 = threadIdx.x + j * kThreads;
    if (i4 < H4) {
      const float4 g = vec4_io<OutT>::load(gain, 4 * (size_t)i4);
      store_act4(h, t, 4 * i4, H,
                 make_float4(v[j].x * r * g.x, v[j].y * r * g.y, v[j].z * r * g.z,
                             v[j].w * r * g.w));
    }
  }
}

// RMSNorm of many rows into the packed bf16 activation layout, 8 rows per
// block: thread tau owns row tau % 8 and the 8-column groups tau / 8 + 128 p
// (p = pass). A store instruction of a wave then covers the 16-byte slots
// of 8 consecutive rows for 8 column groups, i.e. 8 whole 128-byte lines of
// the packed layout (one row per block would write 16 bytes per line and
// leave each line to be completed by 15 other blocks). H % 1024 == 0 and
// H <= 8192 (at most 8 passes held in registers).
__global__ __launch_bounds__(1024) void rmsnorm_rows8_kernel(const float* __restrict__ x, int T,
                                                            int H, bf16_t* __restrict__ h,
                                                            const bf16_t* __restrict__ gain,
                                                            float eps) {
  constexpr int kMaxPass = 8;
  __shared__ float red[16][8];
  const int tau = threadIdx.x, r = tau & 7, kg = tau >> 3;
  const int row = blockIdx.x * 8 + r;
  const bool ok = row < T;
  const int passes = H / 1024;
  float v[kMaxPass][8];
  float ss = 0.f;
#pragma unroll
  for (int p = 0; p < kMaxPass; ++p) {
    if (p < passes) {
      const int k = (p * 128 + kg) * 8;
      float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
      if (ok) {
        a = *(const float4*)(x + (size_t)row * H + k);
        b = *(const float4*)(x + (size_t)row * H + k + 4);
      }
      v[p][0] = a.x; v[p][1] = a.y; v[p][2] = a.z; v[p][3] = a.w;
      v[p][4] = b.x; v[p][5] = b.y; v[p][6] = b.z; v[p][7] = b.w;
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += v[p][e] * v[p][e];
    }
  }
  // lanes with the same row differ in lane bits 3..5, then 16 waves via LDS
  ss += __shfl_xor(ss, 8, 64);
  ss += __shfl_xor(ss, 16, 64);
  ss += __shfl_xor(ss, 32, 64);
  if ((tau & 63) < 8) red[tau >> 6][r] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < 16; ++w) tot += red[w][r];
  if (!ok) return;
  const float sc = 1.0f / sqrtf(tot / (float)H + eps);
#pragma unroll
  for (int p = 0; p < kMaxPass; ++p) {
    if (p < passes) {
      const int k = (p * 128 + kg) * 8;
      const u32x4_t gw = *(const u32x4_t*)(gain + k);
      u32x4_t o;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[e] = pack_bf16x2(v[p][2 * e] * sc * lo_bf16(gw[e]), v[p][2 * e + 1] * sc * hi_bf16(gw[e]));
      *(u32x4_t*)(h + packed_a_offset(row, k, H)) = o;
    }
  }
}

template <typename InT, typename OutT, bool kEmbed, int kThreads>
hipError_t launch_norm_t(const InT* in, const int32_t* rows, float* x, Partials add, OutT* h,
                         const OutT* gain, int T, int H, float eps, hipStream_t s) {
  switch (add.splits) {
#define STAGE_NORM_CASE(S)                                                                  \
  case S:                                                                                   \
    rmsnorm_kernel<InT, OutT, kEmbed, kThreads, S><<<T, kThreads, 0, s>>>(in, rows, x, add.p, \
                                                                         T, add.r0, h, gain, \
                                                                         H, eps);            \
    break;
    STAGE_NORM_CASE(0)
    STAGE_NORM_CASE(1)
    STAGE_NORM_CASE(2)
    STAGE_NORM_CASE(3)
    STAGE_NORM_CASE(4)
    STAGE_NORM_CASE(5)
    STAGE_NORM_CASE(6)
    STAGE_NORM_CASE(7)
    STAGE_NORM_CASE(8)
#undef STAGE_NORM_CASE
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Wide rows get 1024 threads (more loads in flight per row), narrow ones 256.
template <typename InT, typename OutT, bool kEmbed>
hipError_t launch_norm(const InT* in, const int32_t* rows, float* x, Partials add, OutT* h,
                       const OutT* gain, int T, int H, float eps, hipStream_t s) {
  if (H >= 4096)
    return launch_norm_t<InT, OutT, kEmbed, 1024>(in, rows, x, add, h, gain, T, H, eps, s);
  return launch_norm_t<InT, OutT, kEmbed, 256>(in, rows, x, add, h, gain, T, H, eps, s);
}

// Partials cover rows r0 .. T-1 (planes of (T - r0) * H floats).
template <typename OutT>
__global__ __launch_bounds__(256) void output_cast_kernel(const float* __restrict__ x,
                                                          const float* __restrict__ part,
                                                          int splits, int r0, int T, int H,
                                                          OutT* __restrict__ out) {
  const size_t n4 = (size_t)T * H / 4;
  const size_t plane = (size_t)(T - r0) * H, skip = (size_t)r0 * H;
  for (size_t i4 = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i4 < n4;
       i4 += (size_t)gridDim.x * blockDim.x) {
    float4 v = *(const float4*)(x + 4 * i4);
    if (4 * i4 >= skip)
      for (int sp = 0; sp < splits; ++sp)
        add4(v, *(const float4*)(part + sp * plane + 4 * i4 - skip));
    elem<OutT>::store(out, 4 * i4 + 0, v.x);
    elem<OutT>::store(out, 4 * i4 + 1, v.y);
    elem<OutT>::store(out, 4 * i4 + 2, v.z);
    elem<OutT>::store(out, 4 * i4 + 3, v.w);
  }
}

__device__ __forceinline__ const int32_t* seq_table(const SegTables& t, int seq) {
  return seq < t.nseq0 ? t.bt0 + (size_t)seq * t.stride0
                       : t.bt1 + (size_t)(seq - t.nseq0) * t.stride1;
}

// One wave per (TPW consecutive tokens, head); heads [0, n_q)
// are query heads, [n_q, n_q+n_kv) key/value heads. Lane j < d/2 owns the
// rotate-half pair (j, j + d/2). The projection of a column is the sum of
// its source's partial planes. A 1-D grid of (token group, group of 4
// heads) pairs, token group fastest within a head group: first the rows
// t >= r0 (whose source may have several planes, so they are dispatched
// first), then the rows before r0, whose head groups start at g_lo (past
// the query heads when their queries are already rotated). A wave's loads
// for its tokens are independent, so their latency chains (position ->
// rotary table, sequence -> block table) overlap instead of each running in
// a short wave of its own. Steps of a few hundred rows keep one token per
// wave: they need the waves to fill the chip (a decode step of 64 rows has
// 1152), and their sources have several partial planes each.

template <typename T, int TPW>
__global__ __launch_bounds__(256) void rope_kv_kernel(ProjSrc qs, ProjSrc kvs, ProjSrc qt,
                                                      ProjSrc kvt, int r0, int g_lo, int n_tok,
                                                      T* __restrict__ q_out,
                                                      T* __restrict__ kv, int n_kv, int d,
                                                      const int32_t* tok_seq,
                                                      const int32_t* tok_pos, SegTables tabs,
                                                      const float* __restrict__ cos_tab,
                                                      const float* __restrict__ sin_tab,
                                                      const T* __restrict__ q_gain,
                                                      const T* __restrict__ k_gain, float qk_eps,
                                                      int n_q) {
  const int G = (n_q + n_kv + 3) >> 2;  // head groups
  const int nt = n_tok - r0;            // rows from r0 on
  const int ntg = (nt + TPW - 1) / TPW, r0g = (r0 + TPW - 1) / TPW;
  const int wg = blockIdx.x;
  int t0, t_end, grp;
  if (wg < ntg * G) {
    grp = wg / ntg;
    t0 = r0 + (wg % ntg) * TPW;
    t_end = n_tok;
  } else {
    const int w = wg - ntg * G;
    grp = g_lo + w / r0g;
    t0 = (w % r0g) * TPW;
    t_end = r0;
  }
  const int hh = grp * 4 + (threadIdx.x >> 6);
  if (hh >= n_q + n_kv) return;
  const int lane = threadIdx.x & 63;
  const int half = d >> 1;
  const bool act = lane < half;
  const bool is_q = hh < n_q;
  const int kh = hh - n_q;
  const bool tail = t0 >= r0;  // a wave's tokens all lie on one side of r0
  const ProjSrc src = tail ? (is_q ? qt : kvt) : (is_q ? qs : kvs);
  const int col = is_q ? hh * d : kh * d;
  const int vcol = (n_kv + kh) * d;
  const T* gain = is_q ? q_gain : k_gain;

  // Loads for all tokens first (independent, so their latencies overlap);
  // tokens past t_end repeat the last one and are not stored.
  int tt[TPW], pos[TPW];
  const float* row[TPW];
#pragma unroll
  for (int u = 0; u < TPW; ++u) {
    tt[u] = min(t0 + u, t_end - 1);
    pos[u] = tok_pos[tt[u]];
    row[u] = src.base + (size_t)(tail ? tt[u] - r0 : tt[u]) * src.ld;
  }
  float a[TPW], b[TPW], va[TPW], vb[TPW];
#pragma unroll
  for (int u = 0; u < TPW; ++u) a[u] = b[u] = va[u] = vb[u] = 0.f;
  if (act) {
    for (int sp = 0; sp < src.splits; ++sp) {
      const size_t o = (size_t)sp * src.plane;
#pragma unroll
      for (int u = 0; u < TPW; ++u) {
        a[u] += row[u][o + col + lane];
        b[u] += row[u][o + col + lane + half];
        if (!is_q) {
          va[u] += row[u][o + vcol + lane];
          vb[u] += row[u][o + vcol + lane + half];
        }
      }
    }
  }
  if (gain != nullptr) {
    const float ga = act ? elem<T>::load(gain, lane) : 0.f;
    const float gb = act ? elem<T>::load(gain, lane + half) : 0.f;
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
      const float ss = wave_sum(a[u] * a[u] + b[u] * b[u]);
      const float r = 1.0f / sqrtf(ss / (float)d + qk_eps);
      a[u] = a[u] * r * ga;
      b[u] = b[u] * r * gb;
    }
  }
  if (!act) return;
#pragma unroll
  for (int u = 0; u < TPW; ++u) {
    if (t0 + u >= t_end) break;
    const int t = tt[u];
    const float c = cos_tab[(size_t)pos[u] * half + lane];
    const float s = sin_tab[(size_t)pos[u] * half + lane];
    const float ra = a[u] * c - b[u] * s;
    const float rb = a[u] * s + b[u] * c;
    if (is_q) {
      T* qo = q_out + ((size_t)t * n_q + hh) * d;
      elem<T>::store(qo, lane, ra);
      elem<T>::store(qo, lane + half, rb);
      continue;
    }
    const int32_t* bt = seq_table(tabs, tok_seq[t]);
    const int64_t blk = bt[pos[u] / kBlock];
    const int off = pos[u] % kBlock;
    T* kplane = kv + ((blk * n_kv + kh) * 2 + 0) * (int64_t)kBlock * d;
    T* vplane = kplane + (int64_t)kBlock * d;
    elem<T>::store(kplane, kv_k_offset(off, lane), ra);
    elem<T>::store(kplane, kv_k_offset(off, lane + half), rb);
    elem<T>::store(vplane, kv_v_offset(off, lane), va[u]);
    elem<T>::store(vplane, kv_v_offset(off, lane + half), vb[u]);
  }
}

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + expf(-z)); }

__global__ void swiglu_f32_kernel(const float* __restrict__ gu, float* __restrict__ m, int F,
                                  size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x) {
    const size_t t = i / F, j = i % F;
    const float* g = gu + t * 2 * F + j;
    m[i] = silu_f(g[0]) * g[F];
  }
}

// Thread per 4 consecutive output columns c..c+3 of one row; the gate
// columns of the packed gate-up product are (c/32)*64 + c%32, the up
// columns 32 further.
__global__ void swiglu_reduce_kernel(const float* __restrict__ gu, int splits, int T, int F,
                                     bf16_t* __restrict__ m) {
  const size_t plane = (size_t)T * 2 * F;
  const size_t n4 = (size_t)T * F / 4;
  for (size_t i4 = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i4 < n4;
       i4 += (size_t)gridDim.x * blockDim.x) {
    const int t = (int)(i4 / (F / 4));
    const int c = (int)(i4 % (F / 4)) * 4;
    const size_t gcol = (size_t)t * 2 * F + (c / 32) * 64 + (c % 32);
    float4 g = make_float4(0.f, 0.f, 0.f, 0.f), u = g;
    for (int sp = 0; sp < splits; ++sp) {
      add4(g, *(const float4*)(gu + sp * plane + gcol));
      add4(u, *(const float4*)(gu + sp * plane + gcol + 32));
    }
    store_act4(m, t, c, F,
               make_float4(silu_f(g.x) * u.x, silu_f(g.y) * u.y, silu_f(g.z) * u.z,
                           silu_f(g.w) * u.w));
  }
}

inline int grid_for(size_t n, int threads) {
  size_t b = (n + threads - 1) / threads;
  return (int)(b < 8192 ? (b ? b : 1) : 8192);
}

}  // namespace

// Plain streaming copy of n16 16-byte words: each thread moves four words
// per round (loads issued before stores), grid-stride, non-temporal on both
// sides. The known-size reference for bandwidth and hardware traffic
// counters.
__global__ __launch_bounds__(256) void copy_probe_kernel(const u32x4_t* __restrict__ src,
                                                         u32x4_t* __restrict__ dst, size_t n16) {
  const size_t stride = (size_t)gridDim.x * 1024;
  size_t i = (size_t)blockIdx.x * 1024 + threadIdx.x;
  for (; i + 768 < n16; i += stride) {
    u32x4_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = __builtin_nontemporal_load(src + i + u * 256);
#pragma unroll
    for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(v[u], dst + i + u * 256);
  }
  for (; i < n16; i += 256) dst[i] = src[i];
}

hipError_t embed_norm(DType dt, const void* hidden_in, float* x, void* h, const void* gain, int T,
                      int H, float eps, hipStream_t s, const int32_t* rows) {
  if (T == 0) return hipSuccess;
  const Partials none{nullptr, 0};
  if (dt == DT_BF16)
    return launch_norm<bf16_t, bf16_t, true>((const bf16_t*)hidden_in, rows, x, none, (bf16_t*)h,
                                             (const bf16_t*)gain, T, H, eps, s);
  return launch_norm<float, float, true>((const float*)hidden_in, rows, x, none, (float*)h,
                                         (const float*)gain, T, H, eps, s);
}

hipError_t rmsnorm(DType dt, float* x, Partials add, void* h, const void* gain, int T, int H,
                   float eps, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (dt == DT_BF16 && T >= 1024 && H % 1024 == 0 && H <= 8192 &&
      (add.splits == 0 || (add.r0 > 0 && add.r0 % 16 == 0))) {
    // rows with partial sums (a step's last rows) take one row per block,
    // spread over the chip: 8 such rows in one block would read all their
    // planes through one CU
    const int r0 = add.splits ? add.r0 : T;
    if (r0 < T) {
      const hipError_t e = launch_norm<float, bf16_t, false>(
          nullptr, nullptr, x + (size_t)r0 * H, Partials{add.p, add.splits},
          (bf16_t*)h + packed_a_offset(r0, 0, H), (const bf16_t*)gain, T - r0, H, eps, s);
      if (e != hipSuccess) return e;
    }
    rmsnorm_rows8_kernel<<<(r0 + 7) / 8, 1024, 0, s>>>(x, r0, H, (bf16_t*)h, (const bf16_t*)gain,
                                                       eps);
    return hipGetLastError();
  }
  if (dt == DT_BF16)
    return launch_norm<float, bf16_t, false>(nullptr, nullptr, x, add, (bf16_t*)h,
                                             (const bf16_t*)gain, T, H, eps, s);
  return launch_norm<float, float, false>(nullptr, nullptr, x, add, (float*)h, (const float*)gain,
                                          T, H, eps, s);
}

hipError_t output_cast(DType dt, const float* x, Partials add, void* out, int T, int H,
                       hipStream_t s) {
  const size_t n4 = (size_t)T * H / 4;
  if (n4 == 0) return hipSuccess;
  if (dt == DT_BF16)
    output_cast_kernel<bf16_t><<<grid_for(n4, 256), 256, 0, s>>>(x, add.p, add.splits, add.r0,
                                                                 T, H, (bf16_t*)out);
  else
    output_cast_kernel<float><<<grid_for(n4, 256), 256, 0, s>>>(x, add.p, add.splits, add.r0,
                                                                T, H, (float*)out);
  return hipGetLastError();
}

hipError_t rope_kv_write(DType dt, ProjSrc qs, ProjSrc kvs, ProjSrc qt, ProjSrc kvt, int r0,
                         bool q_done, void* q_out, KVLayer kv, const int32_t* tok_seq,
                         const int32_t* tok_pos, SegTables tabs, const float* cos_tab,
                         const float* sin_tab, const void* q_gain, const void* k_gain,
                         float qk_eps, int T, int n_q, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (r0 < 0 || r0 > T) return hipErrorInvalidValue;
  if ((r0 > 0 && (qs.splits < 1 || kvs.splits < 1)) || (r0 < T && (qt.splits < 1 || kvt.splits < 1)))
    return hipErrorInvalidValue;
  if (q_done && n_q % 4 != 0) return hipErrorInvalidValue;
  const int G = (n_q + kv.n_kv + 3) / 4, g_lo = q_done ? n_q / 4 : 0;
  const int tpw = T >= 512 ? 4 : 1;
  dim3 grid((T - r0 + tpw - 1) / tpw * G + (r0 + tpw - 1) / tpw * (G - g_lo));
  auto go = [&](auto elem_tag, auto tpw_c) {
    using E = decltype(elem_tag);
    rope_kv_kernel<E, decltype(tpw_c)::value><<<grid, 256, 0, s>>>(
        qs, kvs, qt, kvt, r0, g_lo, T, (E*)q_out, (E*)kv.base, kv.n_kv, kv.head_dim, tok_seq,
        tok_pos, tabs, cos_tab, sin_tab, (const E*)q_gain, (const E*)k_gain, qk_eps, n_q);
  };
  using One = std::integral_constant<int, 1>;
  using Four = std::integral_constant<int, 4>;
  if (dt == DT_BF16) {
    if (tpw == 4) go(bf16_t{}, Four{}); else go(bf16_t{}, One{});
  } else {
    if (tpw == 4) go(float{}, Four{}); else go(float{}, One{});
  }
  return hipGetLastError();
}

hipError_t swiglu_f32(const float* gu, float* m, int T, int F, hipStream_t s) {
  const size_t n = (size_t)T * F;
  if (n == 0) return hipSuccess;
  swiglu_f32_kernel<<<grid_for(n, 256), 256, 0, s>>>(gu, m, F, n);
  return hipGetLastError();
}

hipError_t swiglu_reduce_bf16(Partials gu, uint16_t* m, int T, int F, hipStream_t s) {
  const size_t n4 = (size_t)T * F / 4;
  if (n4 == 0) return hipSuccess;
  if (gu.r0 != 0) return hipErrorInvalidValue;
  swiglu_reduce_kernel<<<grid_for(n4, 256), 256, 0, s>>>(gu.p, gu.splits, T, F, m);
  return hipGetLastError();
}

hipError_t copy_probe(const void* src, void* dst, size_t bytes, hipStream_t s) {
  const size_t n16 = bytes / 16;
  if (n16 == 0) return hipSuccess;
  const size_t blocks = std::min<size_t>((n16 + 1023) / 1024, 4096);
  copy_probe_kernel<<<(unsigned)blocks, 256, 0, s>>>((const u32x4_t*)src, (u32x4_t*)dst, n16);
  return hipGetLastError();
}

}  // namespace stage_k
