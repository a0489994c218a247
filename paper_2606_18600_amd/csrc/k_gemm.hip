// Linear layers of a decoder layer (QKV, O, gate-up, down):
//   acc[m][n] = sum_k A[m][k] * W[n][k]
// with bf16 operands in the fragment-packed layouts of packed.hpp and fp32
// accumulation on v_mfma_f32_16x16x32_bf16.
//
// * gemm_skinny_bf16: decode-sized M (<= 128). The product is bound by
//   reading W once from HBM. Block = 4 waves on 4 adjacent 64-row groups of W
//   over one K range (the A fragments they share are copied once per block
//   into an LDS ring). Each wave streams its group's fragments (contiguous
//   in the packed layout) with non-temporal loads, two 64-wide k steps in
//   flight, and writes an fp32 partial tile per K split; the consumer
//   kernel sums the splits. With one
//   split the gate-up GEMM applies SwiGLU in its epilogue. 65-128 rows run
//   on 8 waves (gemm_skinny8_bf16); products split over K run on 8 waves
//   over two weight groups and four k parts (gemm_skinny_kp_bf16), which
//   halves the number of partial planes for the same number of blocks.
// * gemm_tiled_bf16: many rows (prefill, mixed steps), compute-bound.
//   256 x 256 (8 waves of 64 x 128), 192 x 256 or 128 x 128 block tiles;
//   weight fragments copied HBM -> LDS with direct loads (64-wide k steps,
//   double-buffered), A fragments loaded straight into registers one or two
//   stages ahead; epilogues: fp32 store, residual add, SwiGLU, query RoPE.
// * gemm_tiled_f32: plain fp32 SIMT tiles (32 or 64 wide) for the fp32 mode
//   (row-major); gemv_f32: fp32 products of at most 8 rows, one wave per
//   output column.
#include <algorithm>
#include <cstdlib>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "packed.hpp"

namespace stage_k {

namespace {

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + expf(-z)); }

// ---------------------------------------------------------------------------
// weight packing
// ---------------------------------------------------------------------------
__global__ void pack_weight_kernel(const bf16_t* __restrict__ src, bf16_t* __restrict__ dst, int N,
                                   int K, int gate_up_ffn) {
  const size_t chunks = (size_t)N * K / 8;
  const int KT = K / 32;
  for (size_t c = blockIdx.x * (size_t)blockDim.x + threadIdx.x; c < chunks;
       c += (size_t)gridDim.x * blockDim.x) {
    const size_t frag = c / 64;
    const int lane = (int)(c % 64);
    const int j = (int)(frag % 4);
    const size_t rest = frag / 4;
    const int g = (int)(rest / KT), kt = (int)(rest % KT);
    const int n = g * 64 + j * 16 + (lane & 15);
    const int k = kt * 32 + (lane >> 4) * 8;
    const int row = gate_up_ffn > 0 ? gate_up_source_row(n, gate_up_ffn) : n;
    *(u32x4_t*)(dst + c * 8) = ldg128(src + (size_t)row * K + k);
  }
}

// ---------------------------------------------------------------------------
// bf16 split-K GEMM for decode-sized M
// ---------------------------------------------------------------------------
constexpr int SK_WAVES = kSkinnyWaves;

enum SkinnyEpi { SK_PARTIAL = 0, SK_SWIGLU = 1 };

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// s_waitcnt immediate that waits until at most n vector-memory operations of
// this wave are outstanding (vmcnt is split over bits 3:0 and 15:14; expcnt
// and lgkmcnt are left at their maxima, i.e. not waited for).
constexpr int vmcnt_at_most(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Block = 4 waves on 4 adjacent 64-column weight groups over the same K
// range. Per 64-wide k step each wave streams its group's 8 W fragments into
// registers (two register sets in ping-pong), while the step's 2*MT A
// fragments, which all four waves need, are copied once per block straight
// into a 3-slot LDS ring (each wave copies a quarter). Streaming the shared
// A through L2 for every wave costs as many bytes as W itself and was the
// limit of this kernel. Every wave issues the same number of loads per step,
// so one vmcnt bound serves all of them.
template <int MT, int EPI>
__global__ __launch_bounds__(SK_WAVES * 64) void gemm_skinny_bf16(const bf16_t* __restrict__ A,
                                                                  const bf16_t* __restrict__ W,
                                                                  int M, int N, int K, int kb_len,
                                                                  void* __restrict__ out) {
  constexpr int NA = (2 * MT + SK_WAVES - 1) / SK_WAVES;  // A copies per wave and step
  constexpr int SLOT = SK_WAVES * NA;                     // fragments per ring slot
  constexpr int WAIT = vmcnt_at_most(8 + NA);             // all but the newest step's loads
  __shared__ u32x4_t As[3][SLOT * 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int G = N / 64;
  const int g_raw = blockIdx.x * SK_WAVES + wave;
  const bool live = g_raw < G;
  // a wave past the last group streams the last group again (and stores
  // nothing) so that it keeps the block's load counts and barriers
  const int g = live ? g_raw : G - 1;
  const int kbeg = blockIdx.y * kb_len;
  const int iters = (min(kb_len, K - kbeg)) / 64;  // >= 1: the grid covers K exactly
  const int r16 = lane & 15;
  const int KT = K / 32;
  const bf16_t* wp = W + ((size_t)g * KT + kbeg / 32) * 4 * 512 + lane * 8;
  // A fragment f = wave + 4u of a step is (m-tile f / 2, k half f % 2); copies
  // past 2*MT re-read the last fragment into slots nobody reads
  const bf16_t* asrc[NA];
#pragma unroll
  for (int u = 0; u < NA; ++u) {
    const int f = min(wave + SK_WAVES * u, 2 * MT - 1);
    asrc[u] = A + ((size_t)(f / 2) * KT + kbeg / 32 + f % 2) * 512 + lane * 8;
  }

  f32x4_t acc[MT][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  u32x4_t wx[2][4], wy[2][4];
  // Loads of k step t. Past the end the index is clamped to the last step:
  // the data is never used, and a copy into the last step's slot writes the
  // bytes that slot already holds.
  auto load = [&](u32x4_t (&w)[2][4], int t) {
    t = t < iters ? t : iters - 1;
    const int slot = t % 3;
#pragma unroll
    for (int u = 0; u < NA; ++u)
      __builtin_amdgcn_global_load_lds((const void*)(asrc[u] + (size_t)t * 2 * 512),
                                       (lds_ptr_t)&As[slot][(wave + SK_WAVES * u) * 64], 16, 0, 0);
    const bf16_t* q = wp + (size_t)t * 8 * 512;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w[h][j] = __builtin_nontemporal_load((const u32x4_t*)(q + (h * 4 + j) * 512));
  };
  auto compute = [&](const u32x4_t (&w)[2][4], int t) {
    const int slot = t % 3;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const u32x4_t a = As[slot][(i * 2 + h) * 64 + lane];
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma16x16x32(a, w[h][j], acc[i][j]);
      }
  };
  // Step t's loads are complete once only step t+1's are outstanding; the
  // barrier then publishes every wave's A copies. Slot (t+2) % 3 is refilled
  // only after the barrier of step t, which every wave reaches after its
  // reads of step t-1 (the slot's previous contents).
  load(wx, 0);
  int t = 0;
  for (; t + 1 < iters; t += 2) {
    load(wy, t + 1);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(WAIT);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    compute(wx, t);
    __builtin_amdgcn_sched_barrier(0);
    load(wx, t + 2);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(WAIT);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    compute(wy, t + 1);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (t < iters) {
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_s_barrier();
    compute(wx, t);
  }
  if (!live) return;

  // C layout of a 16x16 tile: lane l holds column l%16, rows (l/16)*4 + r.
  if (EPI == SK_PARTIAL) {
    float* part = (float*)out + (size_t)blockIdx.y * M * N;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = i * 16 + (lane >> 4) * 4 + r;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) part[(size_t)m * N + g * 64 + j * 16 + r16] = acc[i][j][r];
      }
  } else {
    // tiles 0,1: gate columns 32g..32g+31; tiles 2,3: the matching up columns
    const int F = N / 2;
    bf16_t* mo = (bf16_t*)out;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = i * 16 + (lane >> 4) * 4 + r;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int c = g * 32 + j * 16 + r16;
          mo[packed_a_offset(m, c, F)] = f32_to_bf16(silu_f(acc[i][j][r]) * acc[i][j + 2][r]);
        }
      }
  }
}

// The same product for 65..128 rows with 8 waves per block: wave w streams
// weight group w % 4 and only k tile 2t + w / 4 of each 64-wide step (4 W
// fragments), multiplying it with all MT m-tiles of A from the shared LDS
// ring; the two waves of a group add their sums through LDS at the end and
// each writes half of the m-tiles. A wave's MFMA work per step is then that
// of the 4-wave kernel at 64 rows, and a block runs two waves per SIMD. With
// 128 rows on 4 waves (one per SIMD) the MFMAs of a step took about as long
// as the step's loads, so the two no longer overlapped.
constexpr int SK8_WAVES = 8;

template <int MT, int EPI>
__global__ __launch_bounds__(SK8_WAVES * 64) __attribute__((amdgpu_waves_per_eu(2)))
void gemm_skinny8_bf16(const bf16_t* __restrict__ A, const bf16_t* __restrict__ W, int M, int N,
                       int K, int kb_len, void* __restrict__ out) {
  constexpr int NA = (2 * MT + SK8_WAVES - 1) / SK8_WAVES;  // A copies per wave and step
  constexpr int SLOT = SK8_WAVES * NA;                      // fragments per ring slot
  constexpr int WAIT = vmcnt_at_most(4 + NA);               // all but the newest step's loads
  constexpr int H0 = MT < 4 ? MT : 4;                       // m-tiles [0, H0) end in k half 0
  constexpr int RING = 3 * SLOT * 64;                       // u32x4 of the A ring
  constexpr int RED = 4 * 4 * 4 * 64;                       // u32x4 of one reduction round
  __shared__ u32x4_t lds[RING > RED ? RING : RED];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gw = wave & 3, kh = wave >> 2;
  const int G = N / 64;
  const int g_raw = blockIdx.x * 4 + gw;
  const bool live = g_raw < G;
  const int g = live ? g_raw : G - 1;
  const int kbeg = blockIdx.y * kb_len;
  const int iters = (min(kb_len, K - kbeg)) / 64;  // >= 1: the grid covers K exactly
  const int r16 = lane & 15;
  const int KT = K / 32;
  const bf16_t* wp = W + ((size_t)g * KT + kbeg / 32 + kh) * 4 * 512 + lane * 8;
  const bf16_t* asrc[NA];
#pragma unroll
  for (int u = 0; u < NA; ++u) {
    const int f = min(wave + SK8_WAVES * u, 2 * MT - 1);
    asrc[u] = A + ((size_t)(f / 2) * KT + kbeg / 32 + f % 2) * 512 + lane * 8;
  }

  f32x4_t acc[MT][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  u32x4_t wx[4], wy[4];
  auto load = [&](u32x4_t (&w)[4], int t) {
    t = t < iters ? t : iters - 1;
    const int slot = t % 3;
#pragma unroll
    for (int u = 0; u < NA; ++u)
      __builtin_amdgcn_global_load_lds((const void*)(asrc[u] + (size_t)t * 2 * 512),
                                       (lds_ptr_t)&lds[(slot * SLOT + wave + SK8_WAVES * u) * 64],
                                       16, 0, 0);
    const bf16_t* q = wp + (size_t)t * 8 * 512;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      w[j] = __builtin_nontemporal_load((const u32x4_t*)(q + j * 512));
  };
  auto compute = [&](const u32x4_t (&w)[4], int t) {
    const int slot = t % 3;
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const u32x4_t a = lds[(slot * SLOT + i * 2 + kh) * 64 + lane];
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mfma16x16x32(a, w[j], acc[i][j]);
    }
  };
  // the step loop of gemm_skinny_bf16: step t's loads are complete once only
  // step t+1's are outstanding, and the barrier publishes the A copies
  load(wx, 0);
  int t = 0;
  for (; t + 1 < iters; t += 2) {
    load(wy, t + 1);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(WAIT);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    compute(wx, t);
    __builtin_amdgcn_sched_barrier(0);
    load(wx, t + 2);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(WAIT);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    compute(wy, t + 1);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (t < iters) {
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_s_barrier();
    compute(wx, t);
  }
  // The ring becomes the reduction buffer: every load (the clamped ones past
  // the end included) has landed and every wave has read its last A.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // round 1: k half 1 hands m-tiles [0, H0) to k half 0
  if (kh == 1) {
#pragma unroll
    for (int i = 0; i < H0; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        lds[((gw * 4 + i) * 4 + j) * 64 + lane] = __builtin_bit_cast(u32x4_t, acc[i][j]);
  }
  __syncthreads();
  if (kh == 0) {
#pragma unroll
    for (int i = 0; i < H0; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] += __builtin_bit_cast(f32x4_t, lds[((gw * 4 + i) * 4 + j) * 64 + lane]);
  }
  if constexpr (MT > H0) {
    __syncthreads();
    // round 2: k half 0 hands m-tiles [H0, MT) to k half 1
    if (kh == 0) {
#pragma unroll
      for (int i = H0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          lds[((gw * 4 + i - H0) * 4 + j) * 64 + lane] = __builtin_bit_cast(u32x4_t, acc[i][j]);
    }
    __syncthreads();
    if (kh == 1) {
#pragma unroll
      for (int i = H0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] += __builtin_bit_cast(f32x4_t, lds[((gw * 4 + i - H0) * 4 + j) * 64 + lane]);
    }
  }
  if (!live) return;

  // epilogue of m-tiles [0, H0) (k half 0) or [H0, MT) (k half 1), as in
  // gemm_skinny_bf16
  const int i0 = kh == 0 ? 0 : H0, i1 = kh == 0 ? H0 : MT;
  if (EPI == SK_PARTIAL) {
    float* part = (float*)out + (size_t)blockIdx.y * M * N;
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      if (i < i0 || i >= i1) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = i * 16 + (lane >> 4) * 4 + r;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) part[(size_t)m * N + g * 64 + j * 16 + r16] = acc[i][j][r];
      }
    }
  } else {
    const int F = N / 2;
    bf16_t* mo = (bf16_t*)out;
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      if (i < i0 || i >= i1) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = i * 16 + (lane >> 4) * 4 + r;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int c = g * 32 + j * 16 + r16;
          mo[packed_a_offset(m, c, F)] = f32_to_bf16(silu_f(acc[i][j][r]) * acc[i][j + 2][r]);
        }
      }
    }
  }
}

// Products split over K (splits > 1) on 8 waves as KP = 8 / GW k parts of
// GW adjacent weight groups: wave w streams group w % GW and k tile
// KP t + w / GW of each step t (a step covers 32 KP of K: 4 W fragments per
// wave), multiplying it with all MT m-tiles of A from the shared LDS ring;
// the KP waves of a group add their sums through LDS at the end, each
// finishing MR = ceil(MT / KP) m-tiles. With two groups per block a launch
// needs half the K ranges of the four-group kernels for the same number of
// blocks, so the fp32 partial planes it writes, and its consumer reads,
// halve too.
template <int MT, int GW>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2)))
void gemm_skinny_kp_bf16(const bf16_t* __restrict__ A, const bf16_t* __restrict__ W, int M, int N,
                         int K, int kb_len, float* __restrict__ out, bool rotate) {
  constexpr int KP = 8 / GW;
  constexpr int AF = MT * KP;                        // A fragments per step
  constexpr int NA = (AF + 7) / 8;                   // A copies per wave and step
  constexpr int SLOT = 8 * NA;                       // fragments per ring slot
  constexpr int WAIT = vmcnt_at_most(4 + NA);        // all but the newest step's loads
  constexpr int MR = (MT + KP - 1) / KP;             // m-tiles each wave finishes
  constexpr int RING = 3 * SLOT * 64;                // u32x4 of the A ring
  constexpr int RED = (KP - 1) * GW * MR * 4 * 64;   // u32x4 of one reduction round
  static_assert(GW * KP == 8, "8 waves");
  __shared__ u32x4_t lds[RING > RED ? RING : RED];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gw = wave % GW, kp = wave / GW;
  const int G = N / 64;
  const int g_raw = blockIdx.x * GW + gw;
  const bool live = g_raw < G;
  const int g = live ? g_raw : G - 1;
  const int kbeg = blockIdx.y * kb_len;
  const int iters = (min(kb_len, K - kbeg)) / (32 * KP);  // >= 1: the grid covers K exactly
  const int r16 = lane & 15;
  const int KT = K / 32;
  const bf16_t* wp = W + ((size_t)g * KT + kbeg / 32 + kp) * 4 * 512 + lane * 8;
  // A fragment f of a step is (m-tile f / KP, k tile f % KP); copies past AF
  // re-read the last fragment into slots nobody reads
  const bf16_t* asrc[NA];
#pragma unroll
  for (int u = 0; u < NA; ++u) {
    const int f = min(wave + 8 * u, AF - 1);
    asrc[u] = A + ((size_t)(f / KP) * KT + kbeg / 32 + f % KP) * 512 + lane * 8;
  }

  f32x4_t acc[MT][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  u32x4_t wx[4], wy[4];
  // The block walks its K range from step rot on, wrapping around. The
  // blocks of one K range read the same A fragments; walked in lockstep they
  // ask the same L2 lines at the same moment (batch 128: QKV 45 -> 40, O 37
  // -> 33 us, measured), so each starts at a step of its own.
  const int rot = rotate ? (int)((blockIdx.x * 7u + blockIdx.y * 3u) % (unsigned)iters) : 0;
  // loads of step t, clamped to the last step past the end (as above)
  auto load = [&](u32x4_t (&w)[4], int t) {
    t = t < iters ? t : iters - 1;
    const int slot = t % 3;
    const int ts = t + rot < iters ? t + rot : t + rot - iters;  // the step's data
#pragma unroll
    for (int u = 0; u < NA; ++u)
      __builtin_amdgcn_global_load_lds((const void*)(asrc[u] + (size_t)ts * KP * 512),
                                       (lds_ptr_t)&lds[(slot * SLOT + wave + 8 * u) * 64], 16, 0,
                                       0);
    const bf16_t* q = wp + (size_t)ts * KP * 4 * 512;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      w[j] = __builtin_nontemporal_load((const u32x4_t*)(q + j * 512));
  };
  auto compute = [&](const u32x4_t (&w)[4], int t) {
    const int slot = t % 3;
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const u32x4_t a = lds[(slot * SLOT + i * KP + kp) * 64 + lane];
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mfma16x16x32(a, w[j], acc[i][j]);
    }
  };
  // the step loop of gemm_skinny_bf16
  load(wx, 0);
  int t = 0;
  for (; t + 1 < iters; t += 2) {
    load(wy, t + 1);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(WAIT);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    compute(wx, t);
    __builtin_amdgcn_sched_barrier(0);
    load(wx, t + 2);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(WAIT);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    compute(wy, t + 1);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (t < iters) {
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_s_barrier();
    compute(wx, t);
  }
  // The ring becomes the reduction buffer once every load has landed and
  // every wave has read its last A. Round r: the waves of k parts other than
  // r hand m-tiles [r MR, (r + 1) MR) to the wave of k part r, which adds
  // them in k-part order.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
#pragma unroll
  for (int r = 0; r < KP; ++r) {
    if (r > 0) __syncthreads();
    if (kp != r) {
      const int wr = (kp < r ? kp : kp - 1) * GW + gw;
#pragma unroll
      for (int ii = 0; ii < MR; ++ii) {
        if (r * MR + ii >= MT) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j)
          lds[((wr * MR + ii) * 4 + j) * 64 + lane] = __builtin_bit_cast(u32x4_t, acc[r * MR + ii][j]);
      }
    }
    __syncthreads();
    if (kp == r) {
#pragma unroll
      for (int q = 0; q < KP - 1; ++q) {
        const int wr = q * GW + gw;
#pragma unroll
        for (int ii = 0; ii < MR; ++ii) {
          if (r * MR + ii >= MT) continue;
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[r * MR + ii][j] +=
                __builtin_bit_cast(f32x4_t, lds[((wr * MR + ii) * 4 + j) * 64 + lane]);
        }
      }
    }
  }
  if (!live) return;

  // each wave stores the m-tiles it finished, as in gemm_skinny_bf16
  float* part = out + (size_t)blockIdx.y * M * N;
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    if (i / MR != kp) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = i * 16 + (lane >> 4) * 4 + r;
      if (m >= M) continue;
#pragma unroll
      for (int j = 0; j < 4; ++j) part[(size_t)m * N + g * 64 + j * 16 + r16] = acc[i][j][r];
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 tiled GEMM (prefill / mixed)
// ---------------------------------------------------------------------------
// Block tile: BMT m-tiles (16 rows each) x BNG weight groups (64 columns
// each); waves WM x WN, each owning (BMT/WM) m-tiles x (BNG/WN) groups. One
// stage = 64 of K = 2 k-tiles: BNG*8 W fragments, shared by the WM waves of a
// column, and (BMT/WM)*2 A fragments per wave. The packed layouts make every
// fragment 1 KB contiguous in HBM. The W fragments are copied straight into
// LDS with global_load_lds_dwordx4 (lane l lands at base + 16 l, which is the
// fragment's own lane order), two stages alternating. Each wave loads its A
// fragments straight into registers, a stage ahead, one k-tile half at a
// time: an A fragment feeds 4*(BNG/WN) MFMAs of one wave and at most WN waves
// need it, so staging it in LDS would cost more LDS bandwidth (a write and WN
// reads) than the global load (two L1/L2 hits) it saves.
template <int BMT, int BNG, int WM, int WN, int EPI, bool DEEP>
// DEEP (K ranges of an even number of stages): A is loaded two stages ahead
// into four half-stage register sets in rotation, with loads and copies past
// the end clamped to the last stage, so the stage loop (unrolled by two) has
// no branch and the same wait counts everywhere. Otherwise one stage ahead.
// blockIdx.z selects a K range of k_len (K for an unsplit product) and, for
// the fp32 store, an output plane out + blockIdx.z * out_plane floats.
__global__ __launch_bounds__(WM * WN * 64, 512 / (WM * WN * 64)) void gemm_tiled_bf16(const bf16_t* __restrict__ A,
                                                               const bf16_t* __restrict__ W,
                                                               int M, int N, int K,
                                                               void* __restrict__ out, int ldo,
                                                               int k_len, size_t out_plane,
                                                               RopeRows rope) {
  constexpr int NW = WM * WN;
  constexpr int BF = BNG * 8;
  constexpr int PER_WAVE = BF / NW;
  constexpr int TM = BMT / WM;
  constexpr int TG = BNG / WN;
  static_assert(BF % NW == 0 && BMT % WM == 0 && BNG % WN == 0, "tile split");
  __shared__ u32x4_t lds[2][BF * 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  // Blocks are dealt round-robin to the 8 XCDs (block b -> XCD b % 8), each
  // with its own L2. Remap so that each XCD gets whole weight columns (all
  // m-blocks of a column one after another): a weight tile is then fetched
  // into one L2 instead of all eight. Columns past the last multiple of 8
  // are mapped in plain order.
  int mb, nb;
  {
    const int MB = gridDim.x, NB = gridDim.y, NB8 = NB / 8 * 8;
    const int lin = blockIdx.x + blockIdx.y * MB;
    if (lin < MB * NB8) {
      const int xcd = lin % 8, j = lin / 8;
      nb = (j / MB) * 8 + xcd;
      mb = j % MB;
    } else {
      const int rem = lin - MB * NB8;
      nb = NB8 + rem / MB;
      mb = rem % MB;
    }
  }
  const int mt0 = mb * BMT, g0 = nb * BNG, KT = K / 32;
  const int KTILES = k_len / 64;
  const size_t k0 = (size_t)blockIdx.z * KTILES;  // first stage of this K range

  // this wave's W fragments of a stage: source at stage k0, LDS slot
  const bf16_t* src[PER_WAVE];
#pragma unroll
  for (int p = 0; p < PER_WAVE; ++p) {
    const int fb = wave * PER_WAVE + p;
    src[p] = W + ((((size_t)(g0 + fb / 8) * KT + (fb / 4) % 2) * 4 + fb % 4) + k0 * 8) * 512 + lane * 8;
  }
  auto issue = [&](int kt, int buf) {
#pragma unroll
    for (int p = 0; p < PER_WAVE; ++p)
      __builtin_amdgcn_global_load_lds((const void*)(src[p] + (size_t)kt * 8 * 512),
                                       (lds_ptr_t)&lds[buf][(wave * PER_WAVE + p) * 64], 16, 0, 0);
  };
  // A fragment (m-tile mt0 + wm*TM + i, k-tile 2*(k0 + kt) + h)
  const bf16_t* asrc = A + ((size_t)(mt0 + wm * TM) * KT + 2 * k0) * 512 + lane * 8;
  // The A loads are written as inline asm: the compiler counts direct-to-LDS
  // copies and register loads as completing out of order and would wait for
  // all of them before the first use of an A register. The waits below are
  // explicit instead; each takes the A registers as in/out operands, which
  // keeps their MFMAs after it. Counts: a stage issues PER_WAVE copies and
  // 2*TM A loads, and loads complete in issue order.
  auto aload = [&](u32x4_t (&a)[TM], int kt, int h) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
      asm volatile("global_load_dwordx4 %0, %1, off"
                   : "=v"(a[i])
                   : "v"(asrc + ((size_t)i * KT + 2 * kt + h) * 512)
                   : "memory");
  };
  auto await_a = [&](u32x4_t (&a)[TM], auto n) {
    asm volatile("s_waitcnt vmcnt(%1)" : "+v"(a[0]) : "n"(decltype(n)::value) : "memory");
#pragma unroll
    for (int i = 1; i < TM; ++i) asm volatile("" : "+v"(a[i]));
  };
  using in_flight = std::integral_constant<int, TM + PER_WAVE>;

  f32x4_t acc[TM][TG * 4];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TG * 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  auto half = [&](int buf, int h, const u32x4_t (&a)[TM]) {
    u32x4_t fb[TG * 4];
#pragma unroll
    for (int gi = 0; gi < TG; ++gi)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        fb[gi * 4 + j] = lds[buf][(((wn * TG + gi) * 2 + h) * 4 + j) * 64 + lane];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TG * 4; ++j) acc[i][j] = mfma16x16x32(a[i], fb[j], acc[i][j]);
  };

  if constexpr (DEEP) {
    // Four sets: stage kt uses (sa, sb) = A(kt, h0), A(kt, h1) and reloads
    // them with stage kt + 2. Counts per stage: PER_WAVE copies, 2*TM loads.
    constexpr int AHEAD = 3 * TM + 2 * PER_WAVE;  // issued after A(kt, h)
    const int QMAX = 2 * KTILES - 1;
    auto aload_q = [&](u32x4_t (&a)[TM], int q) {  // half-stage q = 2 kt + h
      q = q < QMAX ? q : QMAX;
#pragma unroll
      for (int i = 0; i < TM; ++i)
        asm volatile("global_load_dwordx4 %0, %1, off"
                     : "=v"(a[i])
                     : "v"(asrc + ((size_t)i * KT + q) * 512)
                     : "memory");
    };
    auto issue_c = [&](int kt, int buf) { issue(kt < KTILES ? kt : KTILES - 1, buf); };
    // weight fragments read per 64-column group: fewer live registers
    auto half_b = [&](int buf, int h, const u32x4_t (&a)[TM]) {
#pragma unroll
      for (int gi = 0; gi < TG; ++gi) {
        u32x4_t fb[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          fb[j] = lds[buf][(((wn * TG + gi) * 2 + h) * 4 + j) * 64 + lane];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][gi * 4 + j] = mfma16x16x32(a[i], fb[j], acc[i][gi * 4 + j]);
      }
    };
    auto stage = [&](int kt, u32x4_t (&sa)[TM], u32x4_t (&sb)[TM]) {
      const int buf = kt & 1;
      issue_c(kt + 1, buf ^ 1);
      await_a(sa, std::integral_constant<int, AHEAD>{});
      half_b(buf, 0, sa);
      aload_q(sa, 2 * kt + 4);
      await_a(sb, std::integral_constant<int, AHEAD>{});
      half_b(buf, 1, sb);
      aload_q(sb, 2 * kt + 5);
      // copies of stage kt + 1 landed (the 2*TM A loads after them may not)
      __builtin_amdgcn_s_waitcnt(vmcnt_at_most(2 * TM));
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
    };
    u32x4_t s0[TM], s1[TM], s2[TM], s3[TM];
    issue(0, 0);
    aload_q(s0, 0);
    aload_q(s1, 1);
    aload_q(s2, 2);
    aload_q(s3, 3);
    await_a(s0, std::integral_constant<int, 0>{});
    await_a(s1, std::integral_constant<int, 0>{});
    await_a(s2, std::integral_constant<int, 0>{});
    await_a(s3, std::integral_constant<int, 0>{});
    __syncthreads();
    for (int kt = 0; kt < KTILES; kt += 2) {
      stage(kt, s0, s1);
      stage(kt + 1, s2, s3);
    }
    // loads past the end still land in the sets: wait before any reuse
    await_a(s0, std::integral_constant<int, 0>{});
    await_a(s1, std::integral_constant<int, 0>{});
    await_a(s2, std::integral_constant<int, 0>{});
    await_a(s3, std::integral_constant<int, 0>{});
  } else {
    u32x4_t a0[TM], a1[TM];  // A of the current stage, k-tile halves 0 and 1
    issue(0, 0);
    aload(a0, 0, 0);
    aload(a1, 0, 1);
    await_a(a0, std::integral_constant<int, 0>{});
    await_a(a1, std::integral_constant<int, 0>{});
    __syncthreads();
    int kt = 0;
    for (; kt + 1 < KTILES; ++kt) {
      const int buf = kt & 1;
      // the other buffer was last read in the previous stage, before its barrier
      issue(kt + 1, buf ^ 1);
      await_a(a0, in_flight{});  // later: a1's loads, this stage's copies
      half(buf, 0, a0);
      aload(a0, kt + 1, 0);
      await_a(a1, in_flight{});  // later: the copies, the new a0 loads
      half(buf, 1, a1);
      aload(a1, kt + 1, 1);
      // the next stage's copies have landed (only the 2*TM A loads issued
      // after them may be in flight); then no wave reads this buffer again
      // (A bare barrier: __syncthreads() would also wait for those A loads.
      // LDS accesses cannot move across it, since the inline asm next to it
      // clobbers memory.)
      __builtin_amdgcn_s_waitcnt(vmcnt_at_most(2 * TM));
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
    }
    await_a(a0, std::integral_constant<int, TM>{});
    half(kt & 1, 0, a0);
    await_a(a1, std::integral_constant<int, 0>{});
    half(kt & 1, 1, a1);
  }

  if (EPI == EPI_STORE_F32 && blockIdx.z != 0) out = (float*)out + blockIdx.z * out_plane;

  // Epilogue: lane l holds column (g*64 + j*16 + l%16), rows (l/16)*4 + r of
  // m-tile (mt0 + wm*TM + i).
  const int r16 = lane & 15;
  if constexpr (EPI == EPI_ROPE_Q) {
    // The wave's two groups are the 128 columns of one head, so both members
    // of each rotate-half pair (jj, jj + 64) are in this lane: tile j of the
    // first group and tile j of the second. With a gain (Qwen3's q RMSNorm)
    // each row is first normalised over the head: the lane's 8 values of the
    // row, then the 16 lanes holding the same rows (lanes 16 q .. 16 q + 15).
    static_assert(TG == 2, "one 128-column head per wave");
    const int hc = (g0 + wn * TG) * 64;  // the head's first column
    const bf16_t* qg = (const bf16_t*)rope.gain;
    float ga[4], gb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      ga[j] = qg ? bf16_to_f32(qg[j * 16 + r16]) : 1.f;
      gb[j] = qg ? bf16_to_f32(qg[64 + j * 16 + r16]) : 1.f;
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float rs = 1.f;
        if (qg) {  // every lane takes part in the shuffles, padding rows too
          float ss = 0.f;
#pragma unroll
          for (int j = 0; j < 8; ++j) ss += acc[i][j][r] * acc[i][j][r];
#pragma unroll
          for (int o = 1; o < 16; o <<= 1) ss += __shfl_xor(ss, o, 64);
          rs = 1.0f / sqrtf(ss / 128.0f + rope.eps);
        }
        const int m = (mt0 + wm * TM + i) * 16 + (lane >> 4) * 4 + r;
        if (m >= M) continue;
        const size_t pr = (size_t)rope.pos[m] * 64;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int jj = j * 16 + r16;
          const float c = rope.cos_tab[pr + jj], sn = rope.sin_tab[pr + jj];
          const float a = acc[i][j][r] * rs * ga[j], b = acc[i][4 + j][r] * rs * gb[j];
          bf16_t* o = (bf16_t*)out + (size_t)m * ldo + hc + jj;
          o[0] = f32_to_bf16(a * c - b * sn);
          o[64] = f32_to_bf16(a * sn + b * c);
        }
      }
    return;
  }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = (mt0 + wm * TM + i) * 16 + (lane >> 4) * 4 + r;
      if (m >= M) continue;
#pragma unroll
      for (int gi = 0; gi < TG; ++gi) {
        const int g = g0 + wn * TG + gi;
        if (EPI == EPI_SWIGLU) {
          // tiles 0,1: gate columns 32g..32g+31; tiles 2,3: the matching up columns;
          // F from ldo, the whole product's width (so a launch may also cover
          // only its first columns)
          const int F = ldo / 2;
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const int c = g * 32 + j * 16 + r16;
            ((bf16_t*)out)[packed_a_offset(m, c, F)] =
                f32_to_bf16(silu_f(acc[i][gi * 4 + j][r]) * acc[i][gi * 4 + j + 2][r]);
          }
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            float* o = (float*)out + (size_t)m * ldo + g * 64 + j * 16 + r16;
            if (EPI == EPI_RESID_ADD)
              *o += acc[i][gi * 4 + j][r];
            else
              *o = acc[i][gi * 4 + j][r];
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// fp32 SIMT tiled GEMM (fp32 mode, row-major operands)
// ---------------------------------------------------------------------------
constexpr int TF_K = 16;

// Block tile TF x TF (64, or 32 when 64-wide tiles would leave most of the
// chip idle), 16 x 16 threads of (TF / 16)^2 outputs each.
template <int TF, int EPI>
__global__ __launch_bounds__(256) void gemm_tiled_f32(const float* __restrict__ A,
                                                      const float* __restrict__ W, int M, int N,
                                                      int K, float* __restrict__ out) {
  constexpr int R = TF / 16;
  __shared__ float As[TF_K][TF + 1];
  __shared__ float Bs[TF_K][TF + 1];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = blockIdx.x * TF, n0 = blockIdx.y * TF;
  float acc[R][R] = {};
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
      float a[R], b[R];
#pragma unroll
      for (int i = 0; i < R; ++i) a[i] = As[c][ty * R + i];
#pragma unroll
      for (int j = 0; j < R; ++j) b[j] = Bs[c][tx * R + j];
#pragma unroll
      for (int i = 0; i < R; ++i)
#pragma unroll
        for (int j = 0; j < R; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int m = m0 + ty * R + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const int n = n0 + tx * R + j;
      if (n >= N) continue;
      if (EPI == EPI_RESID_ADD)
        out[(size_t)m * N + n] += acc[i][j];
      else
        out[(size_t)m * N + n] = acc[i][j];
    }
  }
}

template <int TF>
hipError_t launch_tiled_f32(Epilogue epi, const float* A, const float* W, int M, int N, int K,
                            float* out, hipStream_t s) {
  dim3 grid((M + TF - 1) / TF, (N + TF - 1) / TF);
  if (epi == EPI_RESID_ADD)
    gemm_tiled_f32<TF, EPI_RESID_ADD><<<grid, 256, 0, s>>>(A, W, M, N, K, out);
  else if (epi == EPI_STORE_F32)
    gemm_tiled_f32<TF, EPI_STORE_F32><<<grid, 256, 0, s>>>(A, W, M, N, K, out);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// fp32 products of at most kGemvRows rows (decode steps in the fp32 mode):
// one wave per output column, its lanes striding over K for every row, each
// row's sum then reduced across the wave in a fixed order. On 64 x 64 tiles
// such a product runs N / 64 workgroups over the whole of K (the tiny
// shape's down projection: 4 workgroups, 95 us).
constexpr int kGemvRows = 8;

template <int MR, int EPI>
__global__ __launch_bounds__(256) void gemv_f32(const float* __restrict__ A,
                                                const float* __restrict__ W, int N, int K,
                                                float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const float* w = W + (size_t)n * K;
  float acc[MR];
#pragma unroll
  for (int m = 0; m < MR; ++m) acc[m] = 0.f;
  // unrolled so that several k steps' loads are in flight at once
#pragma unroll 4
  for (int k = lane; k < K; k += 64) {
    const float wk = w[k];
#pragma unroll
    for (int m = 0; m < MR; ++m) acc[m] = fmaf(A[(size_t)m * K + k], wk, acc[m]);
  }
#pragma unroll
  for (int m = 0; m < MR; ++m) {
    const float v = wave_sum(acc[m]);
    if (lane == 0) {
      if (EPI == EPI_RESID_ADD)
        out[(size_t)m * N + n] += v;
      else
        out[(size_t)m * N + n] = v;
    }
  }
}

template <int EPI>
hipError_t launch_gemv_f32(const float* A, const float* W, int M, int N, int K, float* out,
                           hipStream_t s) {
  const int blocks = (N + 3) / 4;
  switch (M) {
    case 1: gemv_f32<1, EPI><<<blocks, 256, 0, s>>>(A, W, N, K, out); break;
    case 2: gemv_f32<2, EPI><<<blocks, 256, 0, s>>>(A, W, N, K, out); break;
    case 3: gemv_f32<3, EPI><<<blocks, 256, 0, s>>>(A, W, N, K, out); break;
    case 4: gemv_f32<4, EPI><<<blocks, 256, 0, s>>>(A, W, N, K, out); break;
    case 5: gemv_f32<5, EPI><<<blocks, 256, 0, s>>>(A, W, N, K, out); break;
    case 6: gemv_f32<6, EPI><<<blocks, 256, 0, s>>>(A, W, N, K, out); break;
    case 7: gemv_f32<7, EPI><<<blocks, 256, 0, s>>>(A, W, N, K, out); break;
    case 8: gemv_f32<8, EPI><<<blocks, 256, 0, s>>>(A, W, N, K, out); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Each block of the k-part kernel walks its K range from a step of its own
// (wrapping around) unless STAGE_SKINNY_ROT=0 (read once).
bool skinny_rot() {
  static const bool on = [] {
    const char* v = getenv("STAGE_SKINNY_ROT");
    return !(v && *v && atoi(v) == 0);
  }();
  return on;
}

// 65..128 rows run on the 8-wave kernel unless STAGE_SKINNY8=0 (read once).
bool skinny8_enabled() {
  static const bool on = [] {
    const char* v = getenv("STAGE_SKINNY8");
    return !(v && *v && atoi(v) == 0);
  }();
  return on;
}

template <int MT>
hipError_t launch_skinny_kp(const bf16_t* a, const bf16_t* w, int M, int N, int K, int kb_len,
                            int splits, void* out, hipStream_t s) {
  const int groups = N / 64;
  dim3 grid((groups + kSkinnyKpGroups - 1) / kSkinnyKpGroups, splits);
  gemm_skinny_kp_bf16<MT, kSkinnyKpGroups><<<grid, 512, 0, s>>>(a, w, M, N, K, kb_len,
                                                                 (float*)out, skinny_rot());
  return hipGetLastError();
}

template <int MT>
hipError_t launch_skinny(const bf16_t* a, const bf16_t* w, int M, int N, int K, int kb_len,
                         bool swiglu, void* out, hipStream_t s) {
  const int groups = N / 64;
  dim3 grid((groups + SK_WAVES - 1) / SK_WAVES, (K + kb_len - 1) / kb_len);
  if constexpr (MT > 4) {
    if (skinny8_enabled()) {
      if (swiglu)
        gemm_skinny8_bf16<MT, SK_SWIGLU><<<grid, SK8_WAVES * 64, 0, s>>>(a, w, M, N, K, kb_len,
                                                                         out);
      else
        gemm_skinny8_bf16<MT, SK_PARTIAL><<<grid, SK8_WAVES * 64, 0, s>>>(a, w, M, N, K, kb_len,
                                                                          out);
      return hipGetLastError();
    }
  }
  if (swiglu)
    gemm_skinny_bf16<MT, SK_SWIGLU><<<grid, SK_WAVES * 64, 0, s>>>(a, w, M, N, K, kb_len, out);
  else
    gemm_skinny_bf16<MT, SK_PARTIAL><<<grid, SK_WAVES * 64, 0, s>>>(a, w, M, N, K, kb_len, out);
  return hipGetLastError();
}

}  // namespace

hipError_t pack_weight(const void* src, void* dst, int N, int K, int gate_up_ffn, hipStream_t s) {
  if (N % 64 != 0 || K % 32 != 0) return hipErrorInvalidValue;
  const size_t chunks = (size_t)N * K / 8;
  size_t blocks = (chunks + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  pack_weight_kernel<<<(int)blocks, 256, 0, s>>>((const bf16_t*)src, (bf16_t*)dst, N, K,
                                                 gate_up_ffn);
  return hipGetLastError();
}

hipError_t gemm_skinny(const void* A, const void* W, int M, int N, int K, int splits,
                       bool swiglu, void* out, hipStream_t s) {
  if (M == 0) return hipSuccess;
  if (M > 128 || N % 64 != 0 || K % 64 != 0 || splits < 1 || (swiglu && splits != 1))
    return hipErrorInvalidValue;
  const bf16_t* a = (const bf16_t*)A;
  const bf16_t* w = (const bf16_t*)W;
  if (skinny_kp_used(K, splits, swiglu)) {
    const int kb = skinny_kp_kb_len(K, splits);
    if ((K + kb - 1) / kb != splits) return hipErrorInvalidValue;  // every split non-empty
    switch ((M + 15) / 16) {
      case 1: return launch_skinny_kp<1>(a, w, M, N, K, kb, splits, out, s);
      case 2: return launch_skinny_kp<2>(a, w, M, N, K, kb, splits, out, s);
      case 3: return launch_skinny_kp<3>(a, w, M, N, K, kb, splits, out, s);
      case 4: return launch_skinny_kp<4>(a, w, M, N, K, kb, splits, out, s);
      case 5: return launch_skinny_kp<5>(a, w, M, N, K, kb, splits, out, s);
      case 6: return launch_skinny_kp<6>(a, w, M, N, K, kb, splits, out, s);
      case 7: return launch_skinny_kp<7>(a, w, M, N, K, kb, splits, out, s);
      default: return launch_skinny_kp<8>(a, w, M, N, K, kb, splits, out, s);
    }
  }
  const int kb = skinny_kb_len(K, splits);
  if ((K + kb - 1) / kb != splits) return hipErrorInvalidValue;  // every split must be non-empty
  switch ((M + 15) / 16) {
    case 1: return launch_skinny<1>(a, w, M, N, K, kb, swiglu, out, s);
    case 2: return launch_skinny<2>(a, w, M, N, K, kb, swiglu, out, s);
    case 3: return launch_skinny<3>(a, w, M, N, K, kb, swiglu, out, s);
    case 4: return launch_skinny<4>(a, w, M, N, K, kb, swiglu, out, s);
    case 5: return launch_skinny<5>(a, w, M, N, K, kb, swiglu, out, s);
    case 6: return launch_skinny<6>(a, w, M, N, K, kb, swiglu, out, s);
    case 7: return launch_skinny<7>(a, w, M, N, K, kb, swiglu, out, s);
    default: return launch_skinny<8>(a, w, M, N, K, kb, swiglu, out, s);
  }
}

// Launch a tiled instantiation, taking the two-stages-ahead A path when the
// K range has an even number of 64-wide stages.
template <int BMT, int BNG, int WM, int WN, int EPI>
void launch_tiled(dim3 grid, hipStream_t s, const bf16_t* A, const bf16_t* W, int M, int N, int K,
                  void* out, int ldo, int k_len, size_t out_plane, RopeRows rope) {
  if ((k_len / 64) % 2 == 0)
    gemm_tiled_bf16<BMT, BNG, WM, WN, EPI, true><<<grid, WM * WN * 64, 0, s>>>(
        A, W, M, N, K, out, ldo, k_len, out_plane, rope);
  else
    gemm_tiled_bf16<BMT, BNG, WM, WN, EPI, false><<<grid, WM * WN * 64, 0, s>>>(
        A, W, M, N, K, out, ldo, k_len, out_plane, rope);
}

hipError_t gemm_split_k(const void* A, const void* W, int M, int N, int K, int splits, float* out,
                        hipStream_t s) {
  if (M == 0) return hipSuccess;
  if (splits < 1 || N % 256 != 0 || K % (64 * splits) != 0) return hipErrorInvalidValue;
  dim3 grid((M + 255) / 256, N / 256, splits);
  launch_tiled<16, 4, 4, 2, EPI_STORE_F32>(grid, s, 
      (const bf16_t*)A, (const bf16_t*)W, M, N, K, out, N, K / splits, (size_t)M * N, RopeRows{});
  return hipGetLastError();
}

// The split-K tail of SwiGLU products (below) unless STAGE_SWIGLU_TAIL_SKINNY=0
// (read once).
bool swiglu_tail_skinny() {
  static const bool on = [] {
    const char* v = getenv("STAGE_SWIGLU_TAIL_SKINNY");
    return !(v && *v && atoi(v) == 0);
  }();
  return on;
}

hipError_t gemm(DType dt, Epilogue epi, const void* A, const void* W, int M, int N, int K,
                void* out, hipStream_t s, RopeRows rope) {
  if (M == 0) return hipSuccess;
  if (epi == EPI_ROPE_Q) {
    // 256 x 256 tiles only: their waves own one 128-column head each
    if (dt != DT_BF16 || N % 256 != 0 || K % 64 != 0 || !rope.pos || !rope.cos_tab ||
        !rope.sin_tab)
      return hipErrorInvalidValue;
    dim3 grid((M + 255) / 256, N / 256);
    launch_tiled<16, 4, 4, 2, EPI_ROPE_Q>(grid, s, 
        (const bf16_t*)A, (const bf16_t*)W, M, N, K, out, N, K, 0, rope);
    return hipGetLastError();
  }
  if (dt == DT_F32 && M <= kGemvRows) {
    if (epi == EPI_RESID_ADD)
      return launch_gemv_f32<EPI_RESID_ADD>((const float*)A, (const float*)W, M, N, K,
                                            (float*)out, s);
    if (epi == EPI_STORE_F32)
      return launch_gemv_f32<EPI_STORE_F32>((const float*)A, (const float*)W, M, N, K,
                                            (float*)out, s);
    return hipErrorInvalidValue;
  }
  if (dt == DT_F32) {
    const long tiles64 = (long)((M + 63) / 64) * ((N + 63) / 64);
    if (tiles64 < 128)
      return launch_tiled_f32<32>(epi, (const float*)A, (const float*)W, M, N, K, (float*)out, s);
    return launch_tiled_f32<64>(epi, (const float*)A, (const float*)W, M, N, K, (float*)out, s);
  }
  if (N % 128 != 0 || K % 64 != 0) return hipErrorInvalidValue;
  // Three tilings: 256 x 256 and 192 x 256 (8 waves, one block per CU) and
  // 128 x 128 (4 waves, two per CU). A product costs about its number of
  // rounds of workgroups times the time of one round. Taking a round of 256
  // 256-row tiles as 1: a round of 256 192-row tiles (3/4 of the work) takes
  // ~0.85 (measured 0.78-0.90), and a round of 512 128 x 128 tiles (half the
  // work, at ~0.97 against ~1.12 PFLOP/s) ~0.58. 192-row tiles win when they
  // fill a round that 256-row tiles leave partly idle (e.g. 2176 x 5120
  // products: 240 tiles instead of 180).
  auto rounds = [](long blocks, long slots) { return (blocks + slots - 1) / slots; };
  const bf16_t* a = (const bf16_t*)A;
  const bf16_t* w = (const bf16_t*)W;
  enum Tiling { T256, T192, T128 };
  // rows [m0, m0 + Ml) and columns [n0, n0 + Nl) of the product: packed A and
  // the packed SwiGLU output start whole 16-row fragments later (m0 % 16 ==
  // 0); fp32 outputs keep the row stride N
  auto launch = [&](Tiling t, int m0, int Ml, int n0, int Nl) -> hipError_t {
    const bf16_t* al = a + (size_t)(m0 / 16) * (K / 32) * 512;
    const bf16_t* wl = w + (size_t)n0 * K;  // packed groups of 64 rows stay in row order
    void* ol = epi == EPI_SWIGLU ? (void*)((bf16_t*)out + (size_t)(m0 / 16) * (N / 64) * 512)
                                 : (void*)((float*)out + (size_t)m0 * N + n0);
    if (t == T256) {
      dim3 grid((Ml + 255) / 256, Nl / 256);
      switch (epi) {
        case EPI_STORE_F32: launch_tiled<16, 4, 4, 2, EPI_STORE_F32>(grid, s, al, wl, Ml, Nl, K, ol, N, K, 0, RopeRows{}); break;
        case EPI_RESID_ADD: launch_tiled<16, 4, 4, 2, EPI_RESID_ADD>(grid, s, al, wl, Ml, Nl, K, ol, N, K, 0, RopeRows{}); break;
        case EPI_SWIGLU: launch_tiled<16, 4, 4, 2, EPI_SWIGLU>(grid, s, al, wl, Ml, Nl, K, ol, N, K, 0, RopeRows{}); break;
        default: return hipErrorInvalidValue;
      }
    } else if (t == T192) {
      dim3 grid((Ml + 191) / 192, Nl / 256);
      switch (epi) {
        case EPI_STORE_F32: launch_tiled<12, 4, 4, 2, EPI_STORE_F32>(grid, s, al, wl, Ml, Nl, K, ol, N, K, 0, RopeRows{}); break;
        case EPI_RESID_ADD: launch_tiled<12, 4, 4, 2, EPI_RESID_ADD>(grid, s, al, wl, Ml, Nl, K, ol, N, K, 0, RopeRows{}); break;
        case EPI_SWIGLU: launch_tiled<12, 4, 4, 2, EPI_SWIGLU>(grid, s, al, wl, Ml, Nl, K, ol, N, K, 0, RopeRows{}); break;
        default: return hipErrorInvalidValue;
      }
    } else {
      dim3 grid((Ml + 127) / 128, Nl / 128);
      switch (epi) {
        case EPI_STORE_F32: launch_tiled<8, 2, 2, 2, EPI_STORE_F32>(grid, s, al, wl, Ml, Nl, K, ol, N, K, 0, RopeRows{}); break;
        case EPI_RESID_ADD: launch_tiled<8, 2, 2, 2, EPI_RESID_ADD>(grid, s, al, wl, Ml, Nl, K, ol, N, K, 0, RopeRows{}); break;
        case EPI_SWIGLU: launch_tiled<8, 2, 2, 2, EPI_SWIGLU>(grid, s, al, wl, Ml, Nl, K, ol, N, K, 0, RopeRows{}); break;
        default: return hipErrorInvalidValue;
      }
    }
    return hipGetLastError();
  };
  auto cost_of = [&](Tiling t, long Ml) -> double {
    if (t == T256) return (double)rounds((Ml + 255) / 256 * (N / 256), 256);
    if (t == T192) return 0.85 * rounds((Ml + 191) / 192 * (N / 256), 256);
    return 0.58 * rounds((Ml + 127) / 128 * (N / 128), 512);
  };
  Tiling best = T128;
  double cost = cost_of(T128, M);
  if (N % 256 == 0) {
    const double c256 = cost_of(T256, M), c192 = cost_of(T192, M);
    if (c192 < cost) best = T192, cost = c192;
    if (c256 <= cost) best = T256, cost = c256;
    const int m1 = M / 256 * 256;
    // A SwiGLU product's rows past the last multiple of 256 (at most 128 of
    // them) on the split-K kernel with one K range and SwiGLU in its
    // epilogue: one more pass over the weights at ~6.3 TB/s, which costs
    // about N / 78000 rounds of 256 x 256 tiles (~5.3 TFLOP/s per CU). Taken
    // when that beats the tilings above, e.g. gate-up at 2048 + 128 rows:
    // -3% at N = 57344 (against the 128 x 128 tail below) and at N = 51200
    // (against 9 partly idle m-blocks), A/B on one box.
    if (epi == EPI_SWIGLU && m1 > 0 && m1 < M && M - m1 <= 128 && swiglu_tail_skinny() &&
        cost_of(T256, m1) + N / 78000.0 < cost) {
      const hipError_t e = launch(T256, 0, m1, 0, N);
      if (e != hipSuccess) return e;
      return gemm_skinny(a + (size_t)(m1 / 16) * (K / 32) * 512, W, M - m1, N, K, 1, true,
                         (bf16_t*)out + (size_t)(m1 / 16) * (N / 64) * 512, s);
    }
    // Otherwise such rows as a launch of their own on 128 x 128 tiles, when
    // the rows before them fill whole rounds of 256-row tiles and the split
    // beats the product on one tiling (-1.3% per 80-layer mixed step before
    // the split-K tail above). Where the first rows would end in a partial
    // round of their own (2048 x 51200: 6.25 rounds) this split measured
    // slower and is not taken.
    if (m1 > 0 && m1 < M && (long)(m1 / 256) * (N / 256) % 256 == 0) {
      const double c_split = cost_of(T256, m1) + cost_of(T128, M - m1);
      if (c_split < cost) {
        const hipError_t e = launch(T256, 0, m1, 0, N);
        if (e != hipSuccess) return e;
        return launch(T128, m1, M - m1, 0, N);
      }
    }
  }
  if (best == T128 && epi != EPI_SWIGLU && N % 256 == 0) {
    // When 256-tiles would leave a partial last round, run the columns that
    // fill whole rounds on 256-tiles and only the rest on 128-tiles.
    long g = (M + 255) / 256, b = 256;
    while (b) { const long t = g % b; g = b; b = t; }  // gcd(m-blocks, 256)
    const long per_round = 256 / g;                     // column blocks per whole round
    const int n1 = (int)((N / 256) / per_round * per_round * 256);
    if (n1 >= N / 2 && n1 < N) {
      const hipError_t e = launch(T256, 0, M, 0, n1);
      if (e != hipSuccess) return e;
      return launch(T128, 0, M, n1, N - n1);
    }
  }
  return launch(best, 0, M, 0, N);
}

}  // namespace stage_k
