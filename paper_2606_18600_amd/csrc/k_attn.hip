// Causal grouped-query attention over the paged KV cache.
//
// Cache geometry per layer: [num_blocks][n_kv][2][16 * d]; plane 0 holds K,
// plane 1 holds V, each as whole 1 KB MFMA operand fragments (kv_k_offset
// and kv_v_offset in packed.hpp).
//
// * attn_decode_bf16: one wave per (decode token, kv head, key split); the 16
//   MFMA rows are the G query heads sharing the kv head (padded to 16).
//     S^T[key][row] = K[key][:] . Q[row][:]        v_mfma_f32_16x16x32_bf16
//     O^T[d][row]  += V^T[d][key] . P^T[key][row]  v_mfma_f32_16x16x16_bf16
//   Every operand is one contiguous fragment load. The C layout of the first
//   product (lane l: row l%16, keys (l/16)*4 + r) is exactly the B layout
//   the second needs, and each lane keeps the online softmax statistics of
//   its own row (4-lane row reductions). Partial (max, sum, unnormalised
//   output) go to a workspace, and attn_merge_kernel combines the splits.
// * attn_prefill_bf16: one 4-wave workgroup per (128 rows of a chunk, kv
//   head); rows are (position, head) pairs of the chunk, keys run from 0 to
//   the last position of the chunk (the chunk's own keys are already in the
//   cache), with the causal mask applied per row. Both products on
//   v_mfma_f32_32x32x16_bf16, with operands gathered per lane from the same
//   fragments (staged in LDS).
// * attn_f32_kernel: plain fp32 SIMT attention, one wave per (token, head),
//   for the fp32 mode.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "packed.hpp"

namespace stage_k {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

// 2^x with the hardware instruction alone. Softmax arguments are <= 8 here
// and results below 2^-126 are negligible next to the row sum, so the
// denormal range handling of exp2f (several more instructions per value, on
// a path bound by these exponentials) is not needed.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
// Online softmax: move the reference maximum only when a block's maximum
// exceeds it by more than this (log2 units).
constexpr float kLazyRescale = 8.0f;

__device__ __forceinline__ const int32_t* seq_table(const SegTables& t, int seq) {
  return seq < t.nseq0 ? t.bt0 + (size_t)seq * t.stride0
                       : t.bt1 + (size_t)(seq - t.nseq0) * t.stride1;
}

// Block ids of a wave's key range are read 64 at a time into one VGPR (lane
// i holds entry w + i) and taken back with v_readlane. A scalar load of each
// entry inside the key loop stalls the loop on every scalar-cache miss before
// the next block's loads can be issued; a conditional refill inside the loop
// makes the compiler wait for all outstanding loads at every readlane. So
// the key loop runs per window: refill, one wait, then the ping-pong over
// the window's blocks.
__device__ __forceinline__ int fill_window(const int32_t* bt, int w, int we, int lane) {
  const int ids = w + lane < we ? bt[w + lane] : 0;
  __builtin_amdgcn_s_waitcnt(0);
  return ids;
}

// K fragments of one 16-token block (kv_k_offset layout): fragment j, lane l
// = token l%16, d = j*32 + (l/16)*8 .. +7; each load reads 1 KB contiguously.
template <int D>
struct KFrag {
  static constexpr int NJ = D / 32;
  u32x4_t v[NJ];
  __device__ __forceinline__ void load(const bf16_t* kplane, int lane) {
    const bf16_t* p = kplane + lane * 8;
#pragma unroll
    for (int j = 0; j < NJ; ++j) v[j] = ldg128(p + j * 512);
  }
  // streaming (non-temporal) variant for data read once
  __device__ __forceinline__ void load_nt(const bf16_t* kplane, int lane) {
    const bf16_t* p = kplane + lane * 8;
#pragma unroll
    for (int j = 0; j < NJ; ++j) v[j] = __builtin_nontemporal_load((const u32x4_t*)(p + j * 512));
  }
};

// V^T fragments of one block (kv_v_offset layout): 1 KB fragment p, lane l
// holds d = 32p + l%16 (words 0-1) and d = 32p + 16 + l%16 (words 2-3), each
// for tokens (l/16)*4 .. +3.
template <int D>
struct VFrag {
  static constexpr int NP = D / 32;
  u32x4_t v[NP];
  __device__ __forceinline__ void load(const bf16_t* vplane, int lane) {
    const bf16_t* p = vplane + lane * 8;
#pragma unroll
    for (int j = 0; j < NP; ++j) v[j] = ldg128(p + j * 512);
  }
  __device__ __forceinline__ void load_nt(const bf16_t* vplane, int lane) {
    const bf16_t* p = vplane + lane * 8;
#pragma unroll
    for (int j = 0; j < NP; ++j) v[j] = __builtin_nontemporal_load((const u32x4_t*)(p + j * 512));
  }
  // A operand of d tile t (16 d values)
  __device__ __forceinline__ u32x2_t tile(int t) const {
    const u32x4_t& w = v[t >> 1];
    return (t & 1) ? u32x2_t{w[2], w[3]} : u32x2_t{w[0], w[1]};
  }
};

// Lanes l, l^16, l^32 and l^48 hold the same row of a 16x16 C tile; combine
// their values with the gfx950 lane swaps (VALU only, no LDS round trip).
// IEEE maximum (NaN-propagating): unlike fmaxf it needs no quieting of its
// operands, and chains of it become three-operand maximum instructions.
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

__device__ __forceinline__ float row4_max(float x) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = vmax(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return vmax(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float row4_sum(float x) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Online-softmax state of the row owned by this lane (row l%16 of a tile).
struct RowState {
  float m, l;
};

// Process one key block for one 16-row tile: scores -> P -> O^T update.
// `s` holds the 4 raw scores (already scaled to log2 units and masked).
template <int D>
__device__ __forceinline__ void softmax_pv(f32x4_t s, RowState& st, f32x4_t* oacc,
                                           const VFrag<D>& vf) {
  const float bm = row4_max(fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3])));
  const float mn = fmaxf(st.m, bm);
  // A row can only be fully masked in a block after an earlier block gave it
  // a finite max, so mn is finite here. (No data-dependent branch here: a
  // branch inside the pipelined key loop makes the compiler wait for every
  // outstanding load at the join.)
  const float alpha = fast_exp2(st.m - mn);
  float p[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) p[r] = fast_exp2(s[r] - mn);
  const float ps = row4_sum(p[0] + p[1] + p[2] + p[3]);
  st.l = st.l * alpha + ps;
  st.m = mn;
  u32x2_t pb;
  pb[0] = pack_bf16x2(p[0], p[1]);
  pb[1] = pack_bf16x2(p[2], p[3]);
#pragma unroll
  for (int t = 0; t < D / 16; ++t) {
    oacc[t] *= alpha;
    oacc[t] = mfma16x16x16(vf.tile(t), pb, oacc[t]);
  }
}

template <int D>
__global__ __launch_bounds__(256) void attn_decode_bf16(const bf16_t* __restrict__ q,
                                                        const bf16_t* __restrict__ kv, int n_kv,
                                                        SegTables tabs,
                                                        const DecodeItem* __restrict__ items,
                                                        const int32_t* __restrict__ order,
                                                        int n_q, float* __restrict__ part_o,
                                                        float* __restrict__ part_ml) {
  const int lane = threadIdx.x & 63;
  const int kvh = blockIdx.y * 4 + (threadIdx.x >> 6);
  if (kvh >= n_kv) return;
  const int idx = order[blockIdx.x];
  const DecodeItem it = items[idx];
  const int G = n_q / n_kv;
  const int row = lane & 15;  // query head within the group
  const bool row_ok = row < G;
  const float scale = kLog2e / sqrtf((float)D);

  // Q^T fragments (B operand): lane l holds head row, same d offsets as K.
  constexpr int NJ = D / 32;
  u32x4_t qf[NJ];
  {
    const bf16_t* qp = q + ((size_t)it.tok * n_q + kvh * G + (row_ok ? row : 0)) * D +
                       (lane >> 4) * 8;
#pragma unroll
    for (int j = 0; j < NJ; ++j) qf[j] = row_ok ? ldg128(qp + j * 32) : u32x4_t{0u, 0u, 0u, 0u};
  }

  const int32_t* bt = seq_table(tabs, it.seq);
  const size_t plane = (size_t)kBlock * D;
  const size_t head_stride = 2 * plane;
  RowState st{-INFINITY, 0.f};
  f32x4_t oacc[D / 16];
#pragma unroll
  for (int t = 0; t < D / 16; ++t) oacc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int b0 = it.k0 / kBlock, b1 = (it.k1 + kBlock - 1) / kBlock;
  // Two register sets in ping-pong (no copies between them), so a block's
  // loads stay in flight while the previous block is processed; the
  // prefetch index is clamped to the window's last block and its data is
  // unused.
  KFrag<D> kx, ky;
  VFrag<D> vx, vy;
  int w = 0, we = 0, ids = 0;
  auto load = [&](KFrag<D>& kf, VFrag<D>& vf, int b) {
    b = b < we ? b : we - 1;
    const bf16_t* kp = kv + ((size_t)__builtin_amdgcn_readlane(ids, b - w) * n_kv + kvh) * head_stride;
    // each (block, kv head) plane is read by exactly one wave of the step:
    // stream it (plain loads that allocate in the caches were ~15% slower)
    kf.load_nt(kp, lane);
    vf.load_nt(kp + plane, lane);
  };
  auto step = [&](const KFrag<D>& kf, const VFrag<D>& vf, int b) {
    f32x4_t s = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < NJ; ++j) s = mfma16x16x32(kf.v[j], qf[j], s);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int key = b * kBlock + (lane >> 4) * 4 + r;
      s[r] = key < it.k1 ? s[r] * scale : -INFINITY;
    }
    softmax_pv<D>(s, st, oacc, vf);
  };
  for (w = b0; w < b1; w += 64) {
    we = min(w + 64, b1);
    ids = fill_window(bt, w, we, lane);
    load(kx, vx, w);
    int b = w;
    for (; b + 1 < we; b += 2) {
      load(ky, vy, b + 1);
      __builtin_amdgcn_sched_barrier(0);
      step(kx, vx, b);
      __builtin_amdgcn_sched_barrier(0);
      load(kx, vx, b + 2);
      __builtin_amdgcn_sched_barrier(0);
      step(ky, vy, b + 1);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (b < we) step(kx, vx, b);
  }

  if (!row_ok) return;
  const size_t ob = ((size_t)idx * n_q + kvh * G + row);
  float* po = part_o + ob * D;
#pragma unroll
  for (int t = 0; t < D / 16; ++t)
    *(f32x4_t*)(po + t * 16 + (lane >> 4) * 4) = oacc[t];
  if (lane < 16) {
    part_ml[ob * 2 + 0] = st.m;
    part_ml[ob * 2 + 1] = st.l;
  }
}

// Combine the key splits of each decode token: one wave per (token, kv
// head). Lane l serves query head row r = l / LPR of the group and DPL
// consecutive d values (a multiple of 4).
template <int D, int G>
__global__ __launch_bounds__(256) void attn_merge_kernel(const float* __restrict__ part_o,
                                                         const float* __restrict__ part_ml,
                                                         const int32_t* __restrict__ item_start,
                                                         const int32_t* __restrict__ tok_rows,
                                                         int n_q, int n_kv,
                                                         bf16_t* __restrict__ out) {
  constexpr int LPR = (64 / G) < (D / 4) ? (64 / G) : (D / 4);  // lanes per head row
  constexpr int DPL = D / LPR;                                    // d values per lane
  const int t = blockIdx.x;
  const int kvh = blockIdx.y * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (kvh >= n_kv || lane >= G * LPR) return;
  const int h = kvh * G + lane / LPR;
  const int d0 = (lane % LPR) * DPL;
  const int i0 = item_start[t], i1 = item_start[t + 1];
  // Online merge over chunks of 4 splits: a chunk's loads are all issued
  // before any is used (indices past the last split are clamped and masked),
  // so a token with up to 4 splits costs one memory round trip.
  float M = -INFINITY, L = 0.f;
  float4 o[DPL / 4];
#pragma unroll
  for (int c = 0; c < DPL / 4; ++c) o[c] = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int i = i0; i < i1; i += 4) {
    float mu[4], lu[4];
    float4 v[4][DPL / 4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const size_t b = (size_t)min(i + u, i1 - 1) * n_q + h;
      mu[u] = part_ml[b * 2];
      lu[u] = part_ml[b * 2 + 1];
      const float4* po = (const float4*)(part_o + b * D + d0);
#pragma unroll
      for (int c = 0; c < DPL / 4; ++c) v[u][c] = po[c];
    }
    float cm = M;
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (i + u < i1) cm = fmaxf(cm, mu[u]);
    const float sc = exp2f(M - cm);  // 0 for the first chunk (M = -inf)
    L *= sc;
#pragma unroll
    for (int c = 0; c < DPL / 4; ++c) {
      o[c].x *= sc;
      o[c].y *= sc;
      o[c].z *= sc;
      o[c].w *= sc;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float w = i + u < i1 ? exp2f(mu[u] - cm) : 0.f;
      L += w * lu[u];
#pragma unroll
      for (int c = 0; c < DPL / 4; ++c) {
        o[c].x += w * v[u][c].x;
        o[c].y += w * v[u][c].y;
        o[c].z += w * v[u][c].z;
        o[c].w += w * v[u][c].w;
      }
    }
    M = cm;
  }
  const float inv = 1.0f / L;
  const int row = tok_rows[t], K = n_q * D;
#pragma unroll
  for (int c = 0; c < DPL / 4; ++c) {
    u32x2_t wv;
    wv[0] = pack_bf16x2(o[c].x * inv, o[c].y * inv);
    wv[1] = pack_bf16x2(o[c].z * inv, o[c].w * inv);
    *(u32x2_t*)(out + packed_a_offset(row, h * D + d0 + 4 * c, K)) = wv;
  }
}

// Prefill: one workgroup of kPfWaves waves per (item, kv head). Row r of
// the workgroup (r < kPfWaves * 32) is query position r / G of the item and
// head kvh*G + r % G; wave w owns rows 32w .. 32w + 31 as one 32-row tile of
// v_mfma_f32_32x32x16_bf16 (lane l: row l % 32). Keys run in stages of BPS
// 16-token blocks: each stage's K and V fragments are copied once into LDS
// (direct loads, two buffers) and read by all waves, so a key is fetched
// once per workgroup instead of once per 32 rows. Scores of a whole stage
// are reduced together; the running maximum is only moved (and the
// accumulators rescaled) when it grows by more than 2^8, so P stays below
// 256 and the rescale is rare after the first stage.
//
// The 32x32x16 form: one wave alone keeps the MFMA pipe nearly full with it
// (2.37 PFLOP/s in a probe, against 1.4 for 16x16x32), which matters here
// because a wave's MFMA work alternates with its softmax arithmetic.
//   S^T[key][row] (32 keys = two blocks x 32 rows): A = K, lane l: key l % 32
//     (block (l / 16) % 2, token l % 16), d 16 ds + 8 (l / 32) .. + 7, read
//     per lane from the blocks' K fragments; B = Q^T, lane l: row l % 32,
//     the same d. C, lane l, value v: row l % 32, key 8 (v / 4) + 4 (l / 32)
//     + v % 4.
//   O^T[d][row] += V^T[d][key] P^T[key][row], 16 keys (one block z of the
//     pair) per product: B = P^T is values 8z .. 8z + 7 of the lane's S^T
//     tile as they stand (k index 8 (l / 32) + e <-> key 8 (e / 4) + 4 (l /
//     32) + e % 4), and A = V^T, lane l: d 32 t + l % 32, the same keys: two
//     8-byte pieces of the block's V fragment t.
constexpr int kPfWaves = 4;
constexpr int kPfBPS = 4;
static_assert(kPfWaves * 32 == kPrefillRows, "rows of a prefill work item");

typedef __attribute__((address_space(3))) void* lds_ptr_t;

__device__ __forceinline__ float row2_max(float x) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return vmax(__uint_as_float(a[0]), __uint_as_float(a[1]));
}
__device__ __forceinline__ float row2_sum(float x) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(a[0]) + __uint_as_float(a[1]);
}

// Two workgroups per CU (64 KB of LDS each) need the register budget of two
// waves per SIMD; one would leave no other wave to overlap a wave's
// exponentials with MFMA work.
template <int D>
__global__ __launch_bounds__(kPfWaves * 64) __attribute__((amdgpu_waves_per_eu(2)))
void attn_prefill_bf16(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kv, int n_kv, SegTables tabs,
    const PrefillItem* __restrict__ items, int n_q, bf16_t* __restrict__ out) {
  constexpr int BPS = kPfBPS;
  constexpr int NJ = D / 32;           // K fragments per block (and V fragments)
  constexpr int FR = 2 * NJ;           // fragments per block
  constexpr int SF = BPS * FR;         // fragments per stage
  constexpr int PER = SF / kPfWaves;   // fragment copies per wave and stage
  constexpr int NP = BPS / 2;          // 32-key tiles per stage
  constexpr int ND = D / 16;           // 16-wide d slices (score products per tile)
  constexpr int NT = D / 32;           // 32-wide d tiles of O^T
  static_assert(SF % kPfWaves == 0, "stage split");
  static_assert(BPS % 2 == 0, "score tiles take key blocks in pairs");
  __shared__ u32x4_t lds[2][SF * 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l32 = lane & 31, hi = lane >> 5;
  // Workgroup b runs on XCD b % 8, each XCD with its own L2. Take the kv head
  // from the linear id modulo n_kv, so every XCD serves a fixed set of kv
  // heads and a sequence's K/V for one head is pulled into one L2 only (not
  // into all eight); items stay in their longest-first order.
  const int lin = blockIdx.x + blockIdx.y * gridDim.x;
  const int kvh = lin % n_kv;
  const PrefillItem it = items[lin / n_kv];
  const int G = n_q / n_kv;
  const float scale = kLog2e / sqrtf((float)D);

  const int r = wave * 32 + l32;  // this lane's row of the workgroup
  const int pi = r / G;
  const bool rok = pi < it.npos;
  const int pc = rok ? pi : it.npos - 1;
  const int rpos = it.p0 + pc;    // its position
  u32x4_t qf[ND];
  {
    const bf16_t* qp = q + ((size_t)(it.t0 + pc) * n_q + kvh * G + r % G) * D + hi * 8;
#pragma unroll
    for (int s = 0; s < ND; ++s) qf[s] = ldg128(qp + s * 16);
  }

  const int32_t* bt = seq_table(tabs, it.seq);
  const size_t plane = (size_t)kBlock * D;
  const int kend = it.p0 + it.npos;  // keys [0, kend)
  const int nb = (kend + kBlock - 1) / kBlock;
  const int nst = (nb + BPS - 1) / BPS;

  RowState st{-INFINITY, 0.f};
  f32x16_t oacc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[t][v] = 0.f;

  // Block ids, 64 at a time (a multiple of BPS, so a stage never straddles
  // two windows).
  int wbase = 0, ids = 0;
  auto issue = [&](int stg, int buf) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int f = wave * PER + p;
      const int c = f % FR;
      int b = stg * BPS + f / FR;
      b = b < nb ? b : nb - 1;  // past the end: a valid block, never used
      const bf16_t* src = kv + ((size_t)__builtin_amdgcn_readlane(ids, b - wbase) * n_kv + kvh) *
                                   (2 * plane) +
                          (c < NJ ? c * 512 : plane + (c - NJ) * 512) + lane * 8;
      __builtin_amdgcn_global_load_lds((const void*)src, (lds_ptr_t)&lds[buf][f * 64], 16, 0, 0);
    }
  };

  // lane offsets inside a block's fragments (u32x4 units): K of d slice s
  // at (s / 2) * 64 + kslot + 32 (s % 2) of block 2 tile + kblk; V pieces
  // at vslot and vslot + 32 (in 8-byte units, half vhalf)
  const int kblk = (lane >> 4) & 1;
  const int kslot = (lane & 15) + 16 * hi;
  const int vslot = (lane & 15) + 16 * hi, vhalf = (lane >> 4) & 1;

  // One stage of BPS key blocks. Stages whose last key is at or before the
  // first query position of the item need no causal mask (for a long
  // context, nearly all of them).
  auto stage = [&](auto masked, int stg) {
    constexpr bool kMask = decltype(masked)::value;
    const int buf = stg & 1;
    if (stg + 1 < nst) {
      if ((stg + 1) * BPS - wbase >= 64) {
        wbase = (stg + 1) * BPS;
        ids = fill_window(bt, wbase, min(wbase + 64, nb), lane);
      }
      issue(stg + 1, buf ^ 1);
    }
    const u32x4_t* L = lds[buf];
    // raw scores of the stage, one 32-key tile per pair of blocks
    f32x16_t sc[NP];
#pragma unroll
    for (int t = 0; t < NP; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) sc[t][v] = 0.f;
#pragma unroll
    for (int s = 0; s < ND; ++s)
#pragma unroll
      for (int t = 0; t < NP; ++t) {
        const u32x4_t kf = L[((2 * t + kblk) * FR + s / 2) * 64 + kslot + 32 * (s % 2)];
        sc[t] = mfma32x32x16(kf, qf[s], sc[t]);
      }
    if constexpr (kMask) {
#pragma unroll
      for (int t = 0; t < NP; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = (stg * BPS + 2 * t) * kBlock + 8 * (v >> 2) + 4 * hi + (v & 3);
          sc[t][v] = key <= rpos ? sc[t][v] : -INFINITY;
        }
    }
    // softmax statistics of the stage (log2 units: score * scale), then P
    float bm = -INFINITY;
#pragma unroll
    for (int t = 0; t < NP; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) bm = vmax(bm, sc[t][v]);
    bm = row2_max(bm) * scale;
    const bool grow = bm > st.m + kLazyRescale;
    const float mn = grow ? bm : st.m;
    const float alpha = fast_exp2(st.m - mn);  // exactly 1 unless the maximum moved
    if (__builtin_amdgcn_ballot_w64(grow) != 0) {
#pragma unroll
      for (int t = 0; t < NT; ++t) oacc[t] *= alpha;
    }
    u32x4_t pb[NP][2];
    float ps = 0.f;
#pragma unroll
    for (int t = 0; t < NP; ++t)
#pragma unroll
      for (int z = 0; z < 2; ++z) {
        float p[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) p[e] = fast_exp2(fmaf(sc[t][8 * z + e], scale, -mn));
        ps += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
        pb[t][z] = u32x4_t{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                           pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])};
      }
    st.l = st.l * alpha + row2_sum(ps);
    st.m = mn;
    // O^T += V^T P^T, block by block. The two 8-byte pieces of each V^T
    // operand are read from LDS straight into adjacent registers (volatile
    // reads, so that the compiler does not merge them with neighbouring
    // pieces and then assemble the operands with register moves).
    typedef const volatile u32x2_t __attribute__((address_space(3)))* lds_u32x2_ptr;
    const lds_u32x2_ptr L2 = (lds_u32x2_ptr)L;
    auto vload = [&](int blk, int t) {
      const int f = blk * FR + NJ + t;
      const u32x2_t a0 = L2[(f * 64 + vslot) * 2 + vhalf];
      const u32x2_t a1 = L2[(f * 64 + vslot + 32) * 2 + vhalf];
      return u32x4_t{a0[0], a0[1], a1[0], a1[1]};
    };
    // Groups g of two products (one block, two d tiles); the V operands of
    // group g + 2 are read while the products of group g run.
    constexpr int NG = BPS * NT / 2, PD = 2;
    u32x4_t va[PD + 1], vb[PD + 1];
    auto vgroup = [&](int g) {
      const int blk = g / (NT / 2), t = 2 * (g % (NT / 2));
      va[g % (PD + 1)] = vload(blk, t);
      vb[g % (PD + 1)] = vload(blk, t + 1);
    };
#pragma unroll
    for (int g = 0; g < PD; ++g) vgroup(g);
    // The compiler's scheduler would otherwise move each read down to just
    // before its product (fewest live registers); these group barriers keep
    // the order: the first PD groups' reads, then per group the reads of
    // group g + PD followed by the products of group g.
    __builtin_amdgcn_sched_group_barrier(0x100, 4 * PD, 0);
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      if (g + PD < NG) vgroup(g + PD);
      const int blk = g / (NT / 2), t = 2 * (g % (NT / 2));
      const u32x4_t pp = pb[blk / 2][blk % 2];
      oacc[t] = mfma32x32x16(va[g % (PD + 1)], pp, oacc[t]);
      oacc[t + 1] = mfma32x32x16(vb[g % (PD + 1)], pp, oacc[t + 1]);
      if (g + PD < NG) __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);  // 4 LDS reads
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);                    // then the MFMAs
    }
    __builtin_amdgcn_s_waitcnt(0);  // the next stage has landed in LDS
    __syncthreads();
  };

  ids = fill_window(bt, 0, min(64, nb), lane);
  issue(0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  const int nfull = min(nst, (it.p0 + 1) / (BPS * kBlock));
  int stg = 0;
  for (; stg < nfull; ++stg) stage(std::false_type{}, stg);
  for (; stg < nst; ++stg) stage(std::true_type{}, stg);

  if (!rok) return;
  const float inv = 1.0f / st.l;
  // packed activation layout (the O projection's input); 4 consecutive
  // columns share one 8-byte piece of a fragment lane
  const int row = it.t0 + pi;
  const int col0 = (kvh * G + r % G) * D + 4 * hi;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int qd = 0; qd < 4; ++qd) {
      u32x2_t w;
      w[0] = pack_bf16x2(oacc[t][4 * qd] * inv, oacc[t][4 * qd + 1] * inv);
      w[1] = pack_bf16x2(oacc[t][4 * qd + 2] * inv, oacc[t][4 * qd + 3] * inv);
      *(u32x2_t*)(out + packed_a_offset(row, col0 + 32 * t + 8 * qd, n_q * D)) = w;
    }
}

// fp32 mode: one wave per (token, query head), keys [0, pos] of its sequence.
// (D is a template argument so that the score and value loops unroll and
// issue their loads ahead of the dependent FMA chains.)
template <int D>
__global__ __launch_bounds__(256) void attn_f32_kernel(const float* __restrict__ q,
                                                       const float* __restrict__ kv, int n_kv,
                                                       SegTables tabs,
                                                       const int32_t* __restrict__ tok_seq,
                                                       const int32_t* __restrict__ tok_pos,
                                                       int t_begin, int n_q,
                                                       float* __restrict__ out) {
  const int t = t_begin + blockIdx.x;
  const int h = blockIdx.y * 4 + (threadIdx.x >> 6);
  if (h >= n_q) return;
  const int lane = threadIdx.x & 63;
  const int kvh = h / (n_q / n_kv);
  const int pos = tok_pos[t];
  const int32_t* bt = seq_table(tabs, tok_seq[t]);
  const float* qp = q + ((size_t)t * n_q + h) * D;
  const float scale = 1.0f / sqrtf((float)D);
  const size_t plane = (size_t)kBlock * D;
  float m = -INFINITY, l = 0.f, o0 = 0.f, o1 = 0.f;
  for (int c0 = 0; c0 <= pos; c0 += 64) {
    const int key = c0 + lane;
    float s = -INFINITY;
    if (key <= pos) {
      const float* kp = kv + ((size_t)bt[key / kBlock] * n_kv + kvh) * 2 * plane;
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < D; ++e) acc = fmaf(qp[e], kp[kv_k_offset(key % kBlock, e)], acc);
      s = acc * scale;
    }
    const float cm = wave_max(s);
    const float mn = fmaxf(m, cm);
    const float alpha = expf(m - mn);
    const float p = key <= pos ? expf(s - mn) : 0.f;
    l = l * alpha + wave_sum(p);
    o0 *= alpha;
    o1 *= alpha;
    auto pv = [&](int j) {
      const float pj = __shfl(p, j, 64);
      const int kj = c0 + j;
      const float* vp = kv + ((size_t)bt[kj / kBlock] * n_kv + kvh) * 2 * plane + plane;
      o0 = fmaf(pj, vp[kv_v_offset(kj % kBlock, lane)], o0);
      if (D > 64) o1 = fmaf(pj, vp[kv_v_offset(kj % kBlock, lane + 64)], o1);
    };
    // whole 64-key chunks unrolled (a loop with a shuffle and a run-time
    // trip count is not), the last partial chunk key by key
    const int nk = min(64, pos + 1 - c0);
    if (nk == 64) {
#pragma unroll 8
      for (int j = 0; j < 64; ++j) pv(j);
    } else {
      for (int j = 0; j < nk; ++j) pv(j);
    }
    m = mn;
  }
  float* op = out + ((size_t)t * n_q + h) * D;
  op[lane] = o0 / l;
  if (D > 64) op[lane + 64] = o1 / l;
}

}  // namespace

hipError_t attn_decode(DType dt, const void* q, KVLayer kv, SegTables tabs,
                       const DecodeItem* items, const int32_t* order, int n_items, int n_q,
                       float* part_o, float* part_ml, hipStream_t s) {
  if (n_items == 0) return hipSuccess;
  if (dt != DT_BF16) return hipErrorInvalidValue;
  dim3 grid(n_items, (kv.n_kv + 3) / 4);
  if (kv.head_dim == 128)
    attn_decode_bf16<128><<<grid, 256, 0, s>>>((const bf16_t*)q, (const bf16_t*)kv.base, kv.n_kv,
                                               tabs, items, order, n_q, part_o, part_ml);
  else if (kv.head_dim == 64)
    attn_decode_bf16<64><<<grid, 256, 0, s>>>((const bf16_t*)q, (const bf16_t*)kv.base, kv.n_kv,
                                              tabs, items, order, n_q, part_o, part_ml);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <int D>
static hipError_t launch_merge(const float* part_o, const float* part_ml, const int32_t* starts,
                               const int32_t* rows, int n_tok, int n_q, int n_kv, bf16_t* out,
                               hipStream_t s) {
  dim3 grid(n_tok, (n_kv + 3) / 4);
  switch (n_q / n_kv) {
    case 1: attn_merge_kernel<D, 1><<<grid, 256, 0, s>>>(part_o, part_ml, starts, rows, n_q, n_kv, out); break;
    case 2: attn_merge_kernel<D, 2><<<grid, 256, 0, s>>>(part_o, part_ml, starts, rows, n_q, n_kv, out); break;
    case 4: attn_merge_kernel<D, 4><<<grid, 256, 0, s>>>(part_o, part_ml, starts, rows, n_q, n_kv, out); break;
    case 8: attn_merge_kernel<D, 8><<<grid, 256, 0, s>>>(part_o, part_ml, starts, rows, n_q, n_kv, out); break;
    case 16: attn_merge_kernel<D, 16><<<grid, 256, 0, s>>>(part_o, part_ml, starts, rows, n_q, n_kv, out); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t attn_merge(DType dt, const float* part_o, const float* part_ml,
                      const int32_t* tok_item_start, const int32_t* tok_rows, int n_tok, int n_q,
                      int n_kv, int head_dim, void* out, hipStream_t s) {
  if (n_tok == 0) return hipSuccess;
  if (dt != DT_BF16) return hipErrorInvalidValue;
  if (head_dim == 128)
    return launch_merge<128>(part_o, part_ml, tok_item_start, tok_rows, n_tok, n_q, n_kv,
                             (bf16_t*)out, s);
  if (head_dim == 64)
    return launch_merge<64>(part_o, part_ml, tok_item_start, tok_rows, n_tok, n_q, n_kv,
                            (bf16_t*)out, s);
  return hipErrorInvalidValue;
}

template <int D>
static void launch_prefill(dim3 grid, hipStream_t s, const void* q, KVLayer kv, SegTables tabs,
                           const PrefillItem* items, int n_q, void* out) {
  attn_prefill_bf16<D><<<grid, kPfWaves * 64, 0, s>>>(
      (const bf16_t*)q, (const bf16_t*)kv.base, kv.n_kv, tabs, items, n_q, (bf16_t*)out);
}

hipError_t attn_prefill(DType dt, const void* q, KVLayer kv, SegTables tabs,
                        const PrefillItem* items, int n_items, int n_q, void* out,
                        hipStream_t s) {
  if (n_items == 0) return hipSuccess;
  if (dt != DT_BF16) return hipErrorInvalidValue;
  if (kPrefillRows % (n_q / kv.n_kv) != 0) return hipErrorInvalidValue;
  dim3 grid(n_items, kv.n_kv);
  if (kv.head_dim == 128)
    launch_prefill<128>(grid, s, q, kv, tabs, items, n_q, out);
  else if (kv.head_dim == 64)
    launch_prefill<64>(grid, s, q, kv, tabs, items, n_q, out);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t attn_f32(const float* q, KVLayer kv, SegTables tabs, const int32_t* tok_seq,
                    const int32_t* tok_pos, int t_begin, int n_tok, int n_q, float* out,
                    hipStream_t s) {
  if (n_tok == 0) return hipSuccess;
  if (kv.head_dim != 64 && kv.head_dim != 128) return hipErrorInvalidValue;
  dim3 grid(n_tok, (n_q + 3) / 4);
  if (kv.head_dim == 128)
    attn_f32_kernel<128><<<grid, 256, 0, s>>>(q, (const float*)kv.base, kv.n_kv, tabs, tok_seq,
                                              tok_pos, t_begin, n_q, out);
  else
    attn_f32_kernel<64><<<grid, 256, 0, s>>>(q, (const float*)kv.base, kv.n_kv, tabs, tok_seq,
                                             tok_pos, t_begin, n_q, out);
  return hipGetLastError();
}

}  // namespace stage_k
