// Linear layers of a decoder layer (QKV, O, gate-up, down):
//   acc[m][n] = sum_k A[m][k] * W[n][k],  A [M,K] row-major, W [N,K] row-major.
//
// * gemm_tiled_bf16: LDS-staged bf16 MFMA tiles (v_mfma_f32_32x32x16_bf16,
//   fp32 accumulate) for steps with many tokens (prefill, mixed), where the
//   products are compute-bound. Fused epilogues: fp32 store, residual add,
//   SwiGLU.
// * gemm_skinny_bf16: split-K weight streaming for decode-sized M, where the
//   product is bound by reading W once from HBM. Each wave streams a 64-row
//   slab of W over one K range and adds its fp32 partial sums atomically.
// * gemm_tiled_f32: plain fp32 SIMT tiles for the fp32 mode.
#include "common.hpp"
#include "kernels.hpp"

namespace stage_k {

namespace {

// ---------------------------------------------------------------------------
// bf16 MFMA tiled GEMM
// ---------------------------------------------------------------------------
constexpr int TB_M = 128, TB_N = 128, TB_K = 64;  // block tile
constexpr int TB_THREADS = 256;                    // 4 waves, 2 x 2, 64 x 64 each
constexpr int TB_CHUNKS = TB_K / 8;                // 16-byte chunks per LDS row

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + expf(-z)); }

template <int EPI>
__global__ __launch_bounds__(TB_THREADS) void gemm_tiled_bf16(const bf16_t* __restrict__ A,
                                                              const bf16_t* __restrict__ W, int M,
                                                              int N, int K, void* __restrict__ out) {
  // LDS rows are TB_K bf16 = 128 B = 8 chunks of 16 B; chunk c of row r is
  // stored at chunk position c ^ (r & 7) so that MFMA fragment reads of 8
  // consecutive rows hit 8 different chunk positions.
  __shared__ u32x4_t As[2][TB_M * TB_CHUNKS];
  __shared__ u32x4_t Bs[2][TB_N * TB_CHUNKS];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.x * TB_M;
  const int nb = blockIdx.y;
  const int half_n = N / 2;  // SwiGLU: gate rows [0, N/2), up rows [N/2, N)

  // Global rows this thread stages (4 chunks of A, 4 of B per K tile).
  const bf16_t* a_src[4];
  const bf16_t* b_src[4];
  int st_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int q = tid + i * TB_THREADS;
    const int r = q >> 3, c = q & 7;
    int am = m0 + r;
    am = am < M ? am : M - 1;
    a_src[i] = A + (size_t)am * K + c * 8;
    int wrow;
    if (EPI == EPI_SWIGLU)
      wrow = (((r >> 5) & 1) ? half_n : 0) + nb * (TB_N / 2) + (r >> 6) * 32 + (r & 31);
    else
      wrow = nb * TB_N + r;
    b_src[i] = W + (size_t)wrow * K + c * 8;
    st_off[i] = r * TB_CHUNKS + (c ^ (r & 7));
  }

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{};

  u32x4_t ra[4], rb[4];
  const int KT = K / TB_K;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ra[i] = ldg128(a_src[i]);
    rb[i] = ldg128(b_src[i]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    As[0][st_off[i]] = ra[i];
    Bs[0][st_off[i]] = rb[i];
  }
  __syncthreads();

  const int frow = lane & 31;   // fragment row within a 32-row tile
  const int fsub = lane >> 5;   // which 8-wide k half of a 16-wide k step
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) {
      const size_t koff = (size_t)(kt + 1) * TB_K;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ra[i] = ldg128(a_src[i] + koff);
        rb[i] = ldg128(b_src[i] + koff);
      }
    }
#pragma unroll
    for (int kk = 0; kk < TB_K / 16; ++kk) {
      const int c = kk * 2 + fsub;
      u32x4_t fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int r = wm * 64 + i * 32 + frow;
        fa[i] = As[buf][r * TB_CHUNKS + (c ^ (r & 7))];
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int r = wn * 64 + j * 32 + frow;
        fb[j] = Bs[buf][r * TB_CHUNKS + (c ^ (r & 7))];
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma32x32x16(fa[i], fb[j], acc[i][j]);
    }
    if (kt + 1 < KT) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        As[buf ^ 1][st_off[i]] = ra[i];
        Bs[buf ^ 1][st_off[i]] = rb[i];
      }
    }
    __syncthreads();
  }

  // Epilogue. Accumulator element e of lane l holds row
  // (e/4)*8 + (l/32)*4 + e%4 and column l%32 of its 32x32 tile.
  const int col = lane & 31;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int m = m0 + wm * 64 + i * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
      if (m >= M) continue;
      if (EPI == EPI_SWIGLU) {
        // tile j=0 holds gate rows, j=1 the matching up rows
        const int n = nb * (TB_N / 2) + wn * 32 + col;
        const float g = acc[i][0][e], u = acc[i][1][e];
        ((bf16_t*)out)[(size_t)m * half_n + n] = f32_to_bf16(silu_f(g) * u);
      } else {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int n = nb * TB_N + wn * 64 + j * 32 + col;
          float* o = (float*)out + (size_t)m * N + n;
          if (EPI == EPI_RESID_ADD)
            *o += acc[i][j][e];
          else
            *o = acc[i][j][e];
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 split-K skinny GEMM (decode)
// ---------------------------------------------------------------------------
// Wave tile: all M rows (MT tiles of 16) x SK_NT tiles of 16 columns, one K
// range. Per 64-wide k step, lane l owns k offsets (l/16)*16 .. +15 of both
// operands (two 16-byte loads), feeding two v_mfma_f32_16x16x32_bf16; the
// reduction over k is order-free, so A and W only need the same mapping.
constexpr int SK_WAVES = 4;

template <int MT, int SK_NT>
__global__ __launch_bounds__(SK_WAVES * 64) void gemm_skinny_bf16(const bf16_t* __restrict__ A,
                                                                  const bf16_t* __restrict__ W,
                                                                  int M, int N, int K, int k_split,
                                                                  float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n0 = (blockIdx.x * SK_WAVES + wave) * (SK_NT * 16);
  if (n0 >= N) return;
  const int kb = blockIdx.y * k_split;
  const int ke = min(K, kb + k_split);
  const int r16 = lane & 15;
  const int koff = (lane >> 4) * 16;

  const bf16_t* wp[SK_NT];
#pragma unroll
  for (int j = 0; j < SK_NT; ++j) wp[j] = W + (size_t)(n0 + j * 16 + r16) * K + koff;
  const bf16_t* ap[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    int m = i * 16 + r16;
    m = m < M ? m : M - 1;
    ap[i] = A + (size_t)m * K + koff;
  }

  f32x4_t acc[MT][SK_NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < SK_NT; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int k = kb; k < ke; k += 64) {
    u32x4_t w0[SK_NT], w1[SK_NT], a0[MT], a1[MT];
#pragma unroll
    for (int j = 0; j < SK_NT; ++j) {
      w0[j] = ldg128(wp[j] + k);
      w1[j] = ldg128(wp[j] + k + 8);
    }
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      a0[i] = ldg128(ap[i] + k);
      a1[i] = ldg128(ap[i] + k + 8);
    }
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < SK_NT; ++j) {
        acc[i][j] = mfma16x16x32(a0[i], w0[j], acc[i][j]);
        acc[i][j] = mfma16x16x32(a1[i], w1[j], acc[i][j]);
      }
  }

  // C layout of a 16x16 tile: lane l holds column l%16, rows (l/16)*4 + r.
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = i * 16 + (lane >> 4) * 4 + r;
      if (m >= M) continue;
#pragma unroll
      for (int j = 0; j < SK_NT; ++j)
        unsafeAtomicAdd(out + (size_t)m * N + n0 + j * 16 + r16, acc[i][j][r]);
    }
}

// ---------------------------------------------------------------------------
// fp32 SIMT tiled GEMM (fp32 mode)
// ---------------------------------------------------------------------------
constexpr int TF = 64, TF_K = 16;

template <int EPI>
__global__ __launch_bounds__(256) void gemm_tiled_f32(const float* __restrict__ A,
                                                      const float* __restrict__ W, int M, int N,
                                                      int K, float* __restrict__ out) {
  __shared__ float As[TF_K][TF + 1];
  __shared__ float Bs[TF_K][TF + 1];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = blockIdx.x * TF, n0 = blockIdx.y * TF;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += TF_K) {
    for (int q = threadIdx.x; q < TF * TF_K; q += 256) {
      const int r = q / TF_K, c = q % TF_K;
      const int m = m0 + r, n = n0 + r, k = k0 + c;
      As[c][r] = (m < M && k < K) ? A[(size_t)m * K + k] : 0.f;
      Bs[c][r] = (n < N && k < K) ? W[(size_t)n * K + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < TF_K; ++c) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[c][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[c][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n >= N) continue;
      if (EPI == EPI_RESID_ADD)
        out[(size_t)m * N + n] += acc[i][j];
      else
        out[(size_t)m * N + n] = acc[i][j];
    }
  }
}

}  // namespace

hipError_t gemm(DType dt, Epilogue epi, const void* A, const void* W, int M, int N, int K,
                void* out, hipStream_t s) {
  if (M == 0) return hipSuccess;
  if (dt == DT_F32) {
    dim3 grid((M + TF - 1) / TF, (N + TF - 1) / TF);
    if (epi == EPI_RESID_ADD)
      gemm_tiled_f32<EPI_RESID_ADD><<<grid, 256, 0, s>>>((const float*)A, (const float*)W, M, N,
                                                          K, (float*)out);
    else if (epi == EPI_STORE_F32)
      gemm_tiled_f32<EPI_STORE_F32><<<grid, 256, 0, s>>>((const float*)A, (const float*)W, M, N,
                                                          K, (float*)out);
    else
      return hipErrorInvalidValue;
    return hipGetLastError();
  }
  if (N % TB_N != 0 || K % TB_K != 0) return hipErrorInvalidValue;
  dim3 grid((M + TB_M - 1) / TB_M, N / TB_N);
  const bf16_t* a = (const bf16_t*)A;
  const bf16_t* w = (const bf16_t*)W;
  switch (epi) {
    case EPI_STORE_F32:
      gemm_tiled_bf16<EPI_STORE_F32><<<grid, TB_THREADS, 0, s>>>(a, w, M, N, K, out);
      break;
    case EPI_RESID_ADD:
      gemm_tiled_bf16<EPI_RESID_ADD><<<grid, TB_THREADS, 0, s>>>(a, w, M, N, K, out);
      break;
    case EPI_SWIGLU:
      gemm_tiled_bf16<EPI_SWIGLU><<<grid, TB_THREADS, 0, s>>>(a, w, M, N, K, out);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int MT, int NT>
static void launch_skinny(const bf16_t* a, const bf16_t* w, int M, int N, int K, int k_split,
                          float* out, hipStream_t s) {
  const int cols_per_block = SK_WAVES * NT * 16;
  dim3 grid((N + cols_per_block - 1) / cols_per_block, (K + k_split - 1) / k_split);
  gemm_skinny_bf16<MT, NT><<<grid, SK_WAVES * 64, 0, s>>>(a, w, M, N, K, k_split, out);
}

hipError_t gemm_skinny(DType dt, const void* A, const void* W, int M, int N, int K, float* out,
                       int k_split, hipStream_t s) {
  if (M == 0) return hipSuccess;
  const int mt = (M + 15) / 16;
  const int nt = mt <= 4 ? 4 : 2;
  if (dt != DT_BF16 || M > 128 || N % (nt * 16) != 0 || K % 64 != 0 || k_split % 64 != 0 ||
      k_split <= 0)
    return hipErrorInvalidValue;
  const bf16_t* a = (const bf16_t*)A;
  const bf16_t* w = (const bf16_t*)W;
  switch (mt) {
    case 1: launch_skinny<1, 4>(a, w, M, N, K, k_split, out, s); break;
    case 2: launch_skinny<2, 4>(a, w, M, N, K, k_split, out, s); break;
    case 3: launch_skinny<3, 4>(a, w, M, N, K, k_split, out, s); break;
    case 4: launch_skinny<4, 4>(a, w, M, N, K, k_split, out, s); break;
    case 5: launch_skinny<5, 2>(a, w, M, N, K, k_split, out, s); break;
    case 6: launch_skinny<6, 2>(a, w, M, N, K, k_split, out, s); break;
    case 7: launch_skinny<7, 2>(a, w, M, N, K, k_split, out, s); break;
    default: launch_skinny<8, 2>(a, w, M, N, K, k_split, out, s); break;
  }
  return hipGetLastError();
}

}  // namespace stage_k
