// Host-side launchers of the stage kernels. Every launcher enqueues on the
// given stream and returns the launch status; none allocates memory.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace stage_k {

enum DType { DT_F32 = 0, DT_BF16 = 1 };

// GEMM epilogues. The GEMM computes acc[m][n] = sum_k A[m][k] * W[n][k]
// (A row-major [M,K], W row-major [N,K]).
enum Epilogue {
  EPI_STORE_F32 = 0,  // out (fp32, [M, N]) = acc
  EPI_RESID_ADD = 1,  // out (fp32 residual, [M, N]) += acc
  EPI_SWIGLU = 2,     // W = [gate (N/2 rows); up (N/2 rows)]; out (mode dtype, [M, N/2]) = silu(g) * u
  EPI_ROPE_Q = 3      // query columns, head_dim 128 (bf16 only): out (bf16, [M, N] row-major) =
                      // rotate-half RoPE of acc at the row's position (RopeRows)
};

// Positions of the rows and the rotary tables ([positions][64] cos and sin)
// for EPI_ROPE_Q.
struct RopeRows {
  const int32_t* pos = nullptr;
  const float* cos_tab = nullptr;
  const float* sin_tab = nullptr;
  const void* gain = nullptr;  // q RMSNorm gain [d] (bf16) before RoPE, or none
  float eps = 0.f;
};

// Block tables of the (at most) two segments of a step: sequences
// [0, nseq0) read table 0, sequences [nseq0, ...) read table 1.
struct SegTables {
  const int32_t* bt0;
  int32_t stride0;
  int32_t nseq0;
  const int32_t* bt1;
  int32_t stride1;
};

// KV cache geometry of one layer: [num_blocks][n_kv][2][block * d]; plane 0
// holds K, plane 1 holds V, in the fragment layouts of packed.hpp.
struct KVLayer {
  void* base;
  int32_t n_kv;
  int32_t head_dim;
};

constexpr int kBlock = 16;

// Decode split-K work item: one decode token attending keys [k0, k1).
struct DecodeItem {
  int32_t tok;  // row of the token in the step
  int32_t seq;  // sequence index (segment-global)
  int32_t k0;
  int32_t k1;
};

// Prefill work item: rows t0 .. t0+npos-1 of one sequence, at positions
// p0 .. p0+npos-1, attending keys [0, p0+npos).
struct PrefillItem {
  int32_t seq;
  int32_t t0;
  int32_t p0;
  int32_t npos;
};

// Split-K partial sums of an fp32 [M, N] result (splits == 0: none). Only
// rows r0 .. M-1 have partials: `splits` planes of (M - r0) * N floats, row
// t at (t - r0) * N of each plane. r0 > 0 when the first r0 rows of a step
// were finished by a tiled product and only the remaining rows ran split-K.
struct Partials {
  const float* p;
  int splits;
  int r0 = 0;
};

// x = fp32(hidden_in); h = RMSNorm(x) * gain. bf16 mode writes h in the packed
// activation layout, fp32 mode row-major. With rows (device, T entries), row t
// of x and h comes from row rows[t] of hidden_in.
hipError_t embed_norm(DType dt, const void* hidden_in, float* x, void* h, const void* gain,
                      int T, int H, float eps, hipStream_t s, const int32_t* rows = nullptr);
// x += sum of the partials; h = RMSNorm(x) * gain (layout as above).
hipError_t rmsnorm(DType dt, float* x, Partials add, void* h, const void* gain, int T, int H,
                   float eps, hipStream_t s);
// out = x + sum of the partials, in the mode dtype, row-major.
hipError_t output_cast(DType dt, const float* x, Partials add, void* out, int T, int H,
                       hipStream_t s);

// Where the fp32 projection feeding RoPE lives: `splits` partial planes of
// `plane` floats each, row t at base + t * ld; the value is the sum over the
// planes. The query columns and the key/value columns are described
// separately (they may come from different products).
struct ProjSrc {
  const float* base;
  int ld;
  int splits;
  size_t plane;
};

// q columns [0, n_q d) from qs, key then value columns [0, 2 n_kv d) from kvs,
// for rows t < r0; rows t >= r0 read row t - r0 of qt and kvt instead (the
// split-K product of a step's last rows; r0 = T: no such rows). With
// q_done, rows t < r0 already have their rotated queries in q_out (the QKV
// product applied RoPE, EPI_ROPE_Q) and only their key/value heads are
// processed (n_q % 4 == 0).
hipError_t rope_kv_write(DType dt, ProjSrc qs, ProjSrc kvs, ProjSrc qt, ProjSrc kvt, int r0,
                         bool q_done, void* q_out, KVLayer kv, const int32_t* tok_seq,
                         const int32_t* tok_pos, SegTables tabs, const float* cos_tab,
                         const float* sin_tab, const void* q_gain, const void* k_gain,
                         float qk_eps, int T, int n_q, hipStream_t s);

// fp32 mode: m = silu(gu[:, :F]) * gu[:, F:] (row-major).
hipError_t swiglu_f32(const float* gu, float* m, int T, int F, hipStream_t s);
// bf16 mode: gu = split-K partials [splits][T][2F] in packed gate-up column
// order; m (packed activation layout [T, F]) = silu(gate) * up.
hipError_t swiglu_reduce_bf16(Partials gu, uint16_t* m, int T, int F, hipStream_t s);

// Pack a row-major bf16 [N, K] weight into the packed layout; gate_up_ffn > 0
// marks the fused gate-up weight (N = 2 * gate_up_ffn).
hipError_t pack_weight(const void* src, void* dst, int N, int K, int gate_up_ffn, hipStream_t s);
// Plain device-to-device copy of `bytes` (a multiple of 16; 16-byte aligned).
hipError_t copy_probe(const void* src, void* dst, size_t bytes, hipStream_t s);

// GEMMs. gemm_skinny (bf16, M <= 128): packed A and W; writes `splits` fp32
// partial planes [splits][M][N] into out, or with swiglu (splits == 1) the
// SwiGLU product in the packed activation layout [M, N/2].
// Split-K partial planes RMSNorm and SwiGLU accept (their loads are unrolled
// over a compile-time count), and the larger number the RoPE / KV-write
// kernel sums in a loop: a narrow QKV projection (one tensor-parallel
// rank's heads) needs many K ranges to occupy the chip.
constexpr int kSkinnyMaxSplits = 8;
// Waves of a split-K decode GEMM workgroup (one 64-row weight group each).
constexpr int kSkinnyWaves = 4;
constexpr int kSkinnyMaxQkvSplits = 32;
// K splits for an [M <= 128] x [N, K] decode GEMM: as many as keep the launch
// at <= target_blocks blocks of 4 waves (at most max_splits).
int skinny_splits(int N, int K, int target_blocks, int max_splits = kSkinnyMaxSplits);
int skinny_kb_len(int K, int splits);
// Products split over K (splits > 1, K % 128 == 0, no SwiGLU) run on the
// k-part kernel: 8 waves on kSkinnyKpGroups weight groups, K ranges a
// multiple of 128, so a launch has half the K ranges of the four-group
// kernels for the same number of blocks. STAGE_SKINNY_KP=0 turns it off
// (read once).
constexpr int kSkinnyKpGroups = 2;
bool skinny_kp_enabled();
bool skinny_kp_used(int K, int splits, bool swiglu);
int skinny_kp_kb_len(int K, int splits);
// K splits for the k-part kernel: as many as keep the launch at
// <= target_blocks blocks (at most max_splits).
int skinny_kp_splits(int N, int K, int target_blocks, int max_splits = kSkinnyMaxSplits);
hipError_t gemm_skinny(const void* A, const void* W, int M, int N, int K, int splits, bool swiglu,
                       void* out, hipStream_t s);
// bf16 LDS-tiled product split over K: `splits` fp32 partial planes
// [splits][M][N] (row stride N) of A [M, K] x W[N, K]^T, 256 x 256 tiles.
// Needs N % 256 == 0 and K % (64 * splits) == 0.
hipError_t gemm_split_k(const void* A, const void* W, int M, int N, int K, int splits, float* out,
                        hipStream_t s);
// gemm: bf16 = LDS-tiled MFMA over packed A and W; fp32 = SIMT, row-major.
hipError_t gemm(DType dt, Epilogue epi, const void* A, const void* W, int M, int N, int K,
                void* out, hipStream_t s, RopeRows rope = RopeRows{});

// Decode attention: workgroup b takes item order[b] (the host's dispatch
// order); partials are written at the item's own index.
hipError_t attn_decode(DType dt, const void* q, KVLayer kv, SegTables tabs,
                       const DecodeItem* items, const int32_t* order, int n_items, int n_q,
                       float* part_o, float* part_ml, hipStream_t s);
hipError_t attn_merge(DType dt, const float* part_o, const float* part_ml,
                      const int32_t* tok_item_start, const int32_t* tok_rows, int n_tok, int n_q,
                      int n_kv, int head_dim, void* out, hipStream_t s);
// Prefill attention: one 4-wave workgroup per (item, kv head), each wave
// holding one tile of 32 (position, head) rows.
hipError_t attn_prefill(DType dt, const void* q, KVLayer kv, SegTables tabs,
                        const PrefillItem* items, int n_items, int n_q, void* out,
                        hipStream_t s);

// fp32 mode: one wave per (token, head) over rows [t_begin, t_begin + n_tok).
hipError_t attn_f32(const float* q, KVLayer kv, SegTables tabs, const int32_t* tok_seq,
                    const int32_t* tok_pos, int t_begin, int n_tok, int n_q, float* out,
                    hipStream_t s);

// (position, head) rows of one prefill attention work item: 4 waves of one
// 32-row tile.
constexpr int kPrefillRows = 128;
// Positions handled by one prefill work item for a GQA group size.
int prefill_item_positions(DType dt, int group);

// Bytes of the library's static device scratch array (one copy per GPU, held
// until the process ends): the workspace of the decode entry point that
// allocates nothing.
constexpr size_t kStaticScratchBytes = (size_t)128 << 20;
// Device address of that array on `device`, which must be the current
// device. Looked up with hipGetSymbolAddress on the first call per device.
hipError_t static_scratch(int device, void** ptr);

// Set the calling thread's message for stage_last_error().
void set_error(const char* msg);

}  // namespace stage_k
