// Row-wise and element-wise kernels of a decoder layer: RMSNorm (with the
// stage-input conversion fused into the first one), per-head q/k RMSNorm +
// RoPE + paged KV write, SwiGLU, and the stage-output cast.
#include "common.hpp"
#include "kernels.hpp"

namespace stage_k {

namespace {

constexpr int kNormThreads = 256;

template <typename InT, typename OutT, bool kEmbed>
__global__ __launch_bounds__(kNormThreads) void rmsnorm_kernel(const InT* __restrict__ in,
                                                               float* __restrict__ x,
                                                               OutT* __restrict__ h,
                                                               const OutT* __restrict__ gain,
                                                               int H, float eps) {
  // One block per row. H is a multiple of 4 (checked by the runtime).
  const size_t row = blockIdx.x;
  __shared__ float red[kNormThreads / STAGE_WAVE];
  float ss = 0.f;
  for (int i = threadIdx.x; i < H; i += kNormThreads) {
    float v;
    if constexpr (kEmbed) {
      v = elem<InT>::load(in, row * H + i);
      x[row * H + i] = v;
    } else {
      v = x[row * H + i];
    }
    ss += v * v;
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kNormThreads / STAGE_WAVE; ++w) tot += red[w];
  const float r = 1.0f / sqrtf(tot / (float)H + eps);
  for (int i = threadIdx.x; i < H; i += kNormThreads) {
    // embed variant: reread the value just written by this same thread
    const float v = x[row * H + i];
    elem<OutT>::store(h, row * H + i, v * r * elem<OutT>::load(gain, i));
  }
}

template <typename OutT>
__global__ void output_cast_kernel(const float* __restrict__ x, OutT* __restrict__ out, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    elem<OutT>::store(out, i, x[i]);
}

__global__ void fill_zero_kernel(float* __restrict__ p, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0.f;
}

__device__ __forceinline__ const int32_t* seq_table(const SegTables& t, int seq) {
  return seq < t.nseq0 ? t.bt0 + (size_t)seq * t.stride0
                       : t.bt1 + (size_t)(seq - t.nseq0) * t.stride1;
}

// One wave per (token, head); heads [0, n_q) are query heads, [n_q, n_q+n_kv)
// key/value heads. Lane j < d/2 owns the rotate-half pair (j, j + d/2).
template <typename T>
__global__ __launch_bounds__(256) void rope_kv_kernel(float* __restrict__ qkv, int zero_after,
                                                      T* __restrict__ q_out, T* __restrict__ kv,
                                                      int n_kv, int d, const int32_t* tok_seq,
                                                      const int32_t* tok_pos, SegTables tabs,
                                                      const float* __restrict__ cos_tab,
                                                      const float* __restrict__ sin_tab,
                                                      const T* __restrict__ q_gain,
                                                      const T* __restrict__ k_gain, float qk_eps,
                                                      int n_q) {
  const int t = blockIdx.x;
  const int hh = blockIdx.y * 4 + (threadIdx.x >> 6);
  if (hh >= n_q + n_kv) return;
  const int lane = threadIdx.x & 63;
  const int half = d >> 1;
  const bool act = lane < half;
  const int pos = tok_pos[t];
  float* row = qkv + (size_t)t * (n_q + 2 * n_kv) * d;
  const bool is_q = hh < n_q;
  const int kh = hh - n_q;
  float* src = is_q ? row + (size_t)hh * d : row + (size_t)(n_q + kh) * d;
  const T* gain = is_q ? q_gain : k_gain;

  float a = act ? src[lane] : 0.f;
  float b = act ? src[lane + half] : 0.f;
  if (gain != nullptr) {
    const float ss = wave_sum(a * a + b * b);
    const float r = 1.0f / sqrtf(ss / (float)d + qk_eps);
    if (act) {
      a = a * r * elem<T>::load(gain, lane);
      b = b * r * elem<T>::load(gain, lane + half);
    }
  }
  if (!act) return;
  const float c = cos_tab[(size_t)pos * half + lane];
  const float s = sin_tab[(size_t)pos * half + lane];
  const float ra = a * c - b * s;
  const float rb = a * s + b * c;
  if (zero_after) {
    src[lane] = 0.f;
    src[lane + half] = 0.f;
  }
  if (is_q) {
    T* qo = q_out + ((size_t)t * n_q + hh) * d;
    elem<T>::store(qo, lane, ra);
    elem<T>::store(qo, lane + half, rb);
    return;
  }
  const int32_t* bt = seq_table(tabs, tok_seq[t]);
  const int64_t blk = bt[pos / kBlock];
  const int off = pos % kBlock;
  T* kplane = kv + ((blk * n_kv + kh) * 2 + 0) * (int64_t)kBlock * d;
  T* vplane = kplane + (int64_t)kBlock * d;
  elem<T>::store(kplane, (size_t)off * d + lane, ra);
  elem<T>::store(kplane, (size_t)off * d + lane + half, rb);
  float* vsrc = row + (size_t)(n_q + n_kv + kh) * d;
  const float va = vsrc[lane], vb = vsrc[lane + half];
  if (zero_after) {
    vsrc[lane] = 0.f;
    vsrc[lane + half] = 0.f;
  }
  elem<T>::store(vplane, (size_t)lane * kBlock + off, va);
  elem<T>::store(vplane, (size_t)(lane + half) * kBlock + off, vb);
}

template <typename T>
__global__ void swiglu_kernel(float* __restrict__ gu, T* __restrict__ m, int F, size_t n,
                              int zero_after) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x) {
    const size_t t = i / F, j = i % F;
    float* g = gu + t * 2 * F + j;
    const float gv = g[0], uv = g[F];
    if (zero_after) {
      g[0] = 0.f;
      g[F] = 0.f;
    }
    elem<T>::store(m, i, gv / (1.0f + expf(-gv)) * uv);
  }
}

inline int grid_for(size_t n, int threads) {
  size_t b = (n + threads - 1) / threads;
  return (int)(b < 8192 ? (b ? b : 1) : 8192);
}

}  // namespace

hipError_t embed_norm(DType dt, const void* hidden_in, float* x, void* h, const void* gain, int T,
                      int H, float eps, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (dt == DT_BF16)
    rmsnorm_kernel<bf16_t, bf16_t, true><<<T, kNormThreads, 0, s>>>(
        (const bf16_t*)hidden_in, x, (bf16_t*)h, (const bf16_t*)gain, H, eps);
  else
    rmsnorm_kernel<float, float, true><<<T, kNormThreads, 0, s>>>(
        (const float*)hidden_in, x, (float*)h, (const float*)gain, H, eps);
  return hipGetLastError();
}

hipError_t rmsnorm(DType dt, const float* x, void* h, const void* gain, int T, int H, float eps,
                   hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (dt == DT_BF16)
    rmsnorm_kernel<float, bf16_t, false><<<T, kNormThreads, 0, s>>>(
        nullptr, const_cast<float*>(x), (bf16_t*)h, (const bf16_t*)gain, H, eps);
  else
    rmsnorm_kernel<float, float, false><<<T, kNormThreads, 0, s>>>(
        nullptr, const_cast<float*>(x), (float*)h, (const float*)gain, H, eps);
  return hipGetLastError();
}

hipError_t output_cast(DType dt, const float* x, void* out, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (dt == DT_BF16)
    output_cast_kernel<bf16_t><<<grid_for(n, 256), 256, 0, s>>>(x, (bf16_t*)out, n);
  else
    output_cast_kernel<float><<<grid_for(n, 256), 256, 0, s>>>(x, (float*)out, n);
  return hipGetLastError();
}

hipError_t fill_zero_f32(float* p, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  fill_zero_kernel<<<grid_for(n, 256), 256, 0, s>>>(p, n);
  return hipGetLastError();
}

hipError_t rope_kv_write(DType dt, float* qkv, int zero_after, void* q_out, KVLayer kv,
                         const int32_t* tok_seq, const int32_t* tok_pos, SegTables tabs,
                         const float* cos_tab, const float* sin_tab, const void* q_gain,
                         const void* k_gain, float qk_eps, int T, int n_q, hipStream_t s) {
  if (T == 0) return hipSuccess;
  dim3 grid(T, (n_q + kv.n_kv + 3) / 4);
  if (dt == DT_BF16)
    rope_kv_kernel<bf16_t><<<grid, 256, 0, s>>>(qkv, zero_after, (bf16_t*)q_out, (bf16_t*)kv.base,
                                                kv.n_kv, kv.head_dim, tok_seq, tok_pos, tabs,
                                                cos_tab, sin_tab, (const bf16_t*)q_gain,
                                                (const bf16_t*)k_gain, qk_eps, n_q);
  else
    rope_kv_kernel<float><<<grid, 256, 0, s>>>(qkv, zero_after, (float*)q_out, (float*)kv.base,
                                               kv.n_kv, kv.head_dim, tok_seq, tok_pos, tabs,
                                               cos_tab, sin_tab, (const float*)q_gain,
                                               (const float*)k_gain, qk_eps, n_q);
  return hipGetLastError();
}

hipError_t swiglu(DType dt, float* gu, void* m, int T, int F, int zero_after, hipStream_t s) {
  const size_t n = (size_t)T * F;
  if (n == 0) return hipSuccess;
  if (dt == DT_BF16)
    swiglu_kernel<bf16_t><<<grid_for(n, 256), 256, 0, s>>>(gu, (bf16_t*)m, F, n, zero_after);
  else
    swiglu_kernel<float><<<grid_for(n, 256), 256, 0, s>>>(gu, (float*)m, F, n, zero_after);
  return hipGetLastError();
}

}  // namespace stage_k
