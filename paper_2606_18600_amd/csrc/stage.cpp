// Stage runtime: argument validation, workspace planning, per-step metadata
// and the per-layer launch sequence behind the C ABI of include/stage.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/stage.h"
#include "kernels.hpp"

using namespace stage_k;

namespace {

thread_local std::string g_err;
std::atomic<uint64_t> g_stage_uid{0};

// Per device: the stage whose call last used the static scratch array (its
// uid; 0 = none). Only that stage's rotary table is known to be there.
constexpr int kMaxStaticDevices = 64;
std::mutex g_static_mu;
uint64_t g_static_owner[kMaxStaticDevices] = {};

stage_status fail(stage_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

constexpr int kRing = 4;             // pinned staging buffers in flight
constexpr int kMaxSplits = 32;       // decode key splits per sequence, at most
constexpr int kSplitMinBlocks = 4;   // at least 4 blocks (64 keys) per split
constexpr int kSkinnyMaxRows = 128;  // decode-sized steps use split-K GEMMs
constexpr int kMaxKvSplits = 4;      // K splits of the key/value columns of a prefill QKV
constexpr int kMaxMidSplits = 8;     // K splits of the products of a small tiled step
constexpr int kMidRows = 2048;       // partial-plane rows of such a step (splits x T) ...
constexpr size_t kMidElems = 16u << 20;  // ... or this many fp32 values, if more (narrow N)

// fp32 values the partial planes of a small tiled step's [T, N] product may
// take (T <= max_tokens): kMidRows rows, or for narrow products (tensor-
// parallel shards, whose 256-wide tiles need more K ranges to fill a round)
// up to kMidElems values, as far as kMaxMidSplits planes of max_tokens rows
// need them.
size_t mid_capacity(int max_tokens, int N) {
  return std::max((size_t)kMidRows * N,
                  std::min(kMidElems, (size_t)kMaxMidSplits * max_tokens * N));
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Decode split items of a step, at most. The plan (build_meta) aims at
// `attn_waves` waves: with u = sum over sequences of their key blocks, every
// split covers at least ceil(n_kv u / attn_waves) blocks, so sequence j gets
// ceil(nb_j / bps) < nb_j / bps + 1 splits and the step fewer than
// attn_waves / n_kv + (sequences) in total.
size_t max_decode_items(int max_seqs, int attn_waves, int n_kv) {
  const size_t by_plan = (size_t)max_seqs + (size_t)((attn_waves + n_kv - 1) / n_kv);
  return std::min((size_t)max_seqs * kMaxSplits, by_plan);
}

// The waves a decode step of nd sequences aims for: attn_waves up to 64
// sequences, then half as much again per 128 more (measured on the
// Llama-70B shape: 1600 best at 64 sequences, 2400 at 128, where 1600 and
// 3200 were 1.4% and 1.3% slower).
int decode_waves(int attn_waves, int nd, bool scale) {
  if (!scale || nd <= 64) return attn_waves;
  return (int)((long long)attn_waves * (128 + nd - 64) / 128);
}

int env_int(const char* name, int dflt) {
  const char* v = getenv(name);
  return (v && *v) ? atoi(v) : dflt;
}

struct Region {
  size_t off = 0, bytes = 0;
};

struct PendingTiming {
  int op;
  hipEvent_t e0, e1;
};

}  // namespace

void stage_k::set_error(const char* msg) { g_err = msg ? msg : ""; }

struct stage {
  stage_model_config cfg{};
  int32_t layer_begin = 0, n_layers = 0;
  std::vector<stage_layer_weights> layers;
  char* kv_pool = nullptr;
  int32_t num_blocks = 0;
  int32_t max_tokens = 0, max_seqs = 0;
  size_t esize = 4;
  size_t kv_layer_bytes = 0;
  int device = 0;
  int skinny_rows = 0;  // steps with at most this many tokens use split-K GEMMs
  // K splits of the four split-K GEMMs (QKV, O, gate-up, down)
  int s_qkv = 1, s_o = 1, s_gu = 1, s_down = 1;
  // decode attention waves to aim for: one resident round (the kernel runs
  // two waves per SIMD, 2048 on the chip) with slack for per-sequence
  // rounding of the split sizes
  int cus = 256;  // compute units of the device
  int attn_waves = 1600;
  bool attn_scale = true;  // more decode attention waves for batches above 64
  bool row_tail_on = true;  // split-K skinny products for the last rows of large steps
  bool q_rope_fused = true;  // RoPE in the epilogue of a step's query product (when possible)
  bool q_norm_fused = true;  // ... also after a q RMSNorm (q/k-norm models)
  bool check_tables = false;  // copy block tables to the host and check ids (STAGE_DEBUG)

  uint64_t uid = 0;        // distinct for every stage created in the process
  size_t max_ditems = 0;   // decode split items a step may need (bf16)
  // rotary table (angle p * theta^(-2j/d) in double, rounded once to float),
  // [max_position][head_dim / 2] cos then sin; uploaded into the workspace
  std::vector<float> rope_host;

  // workspace
  Region r_x, r_h, r_qkv, r_kvpart, r_q, r_attn, r_m, r_gu, r_part_x, r_part_o, r_part_ml, r_meta,
      r_cos, r_sin;
  size_t ws_bytes = 0;
  char* ws = nullptr;
  size_t meta_ints = 0;

  // pinned staging ring for per-step metadata
  int32_t* staging[kRing] = {};
  hipEvent_t staging_ev[kRing] = {};
  bool staging_used[kRing] = {};
  int ring = 0;

  // op timing
  bool timing = false;
  std::vector<PendingTiming> pending;
  std::vector<hipEvent_t> free_events;
  double op_ms[STAGE_OP_COUNT] = {};
  int64_t op_launches[STAGE_OP_COUNT] = {};

  template <typename T>
  T* at(const Region& r) const {
    return reinterpret_cast<T*>(ws + r.off);
  }
};

namespace {

bool is_pow2_le16(int g) { return g == 1 || g == 2 || g == 4 || g == 8 || g == 16; }

stage_status check_config(const stage_model_config* c) {
  if (!c) return fail(STAGE_ERR_INVALID_ARG, "config is NULL");
  if (c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 ||
      c->ffn <= 0 || c->max_position <= 0)
    return fail(STAGE_ERR_INVALID_ARG, "config sizes must be positive");
  if (!(c->rms_eps >= 0.f) || !(c->qk_rms_eps >= 0.f) || !(c->rope_theta > 0.0))
    return fail(STAGE_ERR_INVALID_ARG, "eps must be >= 0 and rope_theta > 0");
  // A C caller can store any integer in the enum field: read it as one.
  static_assert(sizeof(stage_dtype) == sizeof(int32_t), "stage_dtype is a 32-bit enum");
  int32_t dtype_raw;
  std::memcpy(&dtype_raw, &c->dtype, sizeof dtype_raw);
  if (dtype_raw != STAGE_F32 && dtype_raw != STAGE_BF16)
    return fail(STAGE_ERR_UNSUPPORTED, "dtype %d not supported", (int)dtype_raw);
  if (c->block_size != kBlock)
    return fail(STAGE_ERR_UNSUPPORTED, "block_size must be %d (got %d)", kBlock, c->block_size);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(STAGE_ERR_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", c->head_dim);
  if (c->n_q_heads % c->n_kv_heads != 0 || !is_pow2_le16(c->n_q_heads / c->n_kv_heads))
    return fail(STAGE_ERR_UNSUPPORTED, "n_q_heads/n_kv_heads must be 1, 2, 4, 8 or 16");
  if (c->hidden > 16384)
    return fail(STAGE_ERR_UNSUPPORTED, "hidden %d > 16384", c->hidden);
  if (c->hidden % 128 != 0 || (c->n_q_heads * c->head_dim) % 128 != 0 || c->ffn % 64 != 0)
    return fail(STAGE_ERR_UNSUPPORTED,
                "need hidden %% 128 == 0, n_q*head_dim %% 128 == 0, ffn %% 64 == 0");
  if (c->qk_norm != 0 && c->qk_norm != 1)
    return fail(STAGE_ERR_INVALID_ARG, "qk_norm must be 0 or 1");
  return STAGE_OK;
}

// Validate one batch against the stage limits; `decode` requires q_len == 1.
stage_status check_batch(const stage_model_config& c, const stage_batch* b, bool decode,
                         const char* what, long long* tokens) {
  *tokens = 0;
  if (!b || b->num_seqs == 0) return STAGE_OK;
  if (b->num_seqs < 0) return fail(STAGE_ERR_INVALID_ARG, "%s: num_seqs < 0", what);
  if (!b->q_lens || !b->ctx_lens)
    return fail(STAGE_ERR_INVALID_ARG, "%s: q_lens/ctx_lens is NULL", what);
  if (!b->block_tables) return fail(STAGE_ERR_INVALID_ARG, "%s: block_tables is NULL", what);
  if (b->max_blocks_per_seq <= 0)
    return fail(STAGE_ERR_INVALID_ARG, "%s: max_blocks_per_seq must be >= 1", what);
  const long long cap = (long long)b->max_blocks_per_seq * c.block_size;
  for (int i = 0; i < b->num_seqs; ++i) {
    const long long q = b->q_lens[i], ctx = b->ctx_lens[i];
    if (q < 1) return fail(STAGE_ERR_INVALID_ARG, "%s: q_lens[%d] = %lld < 1", what, i, q);
    if (decode && q != 1)
      return fail(STAGE_ERR_INVALID_ARG, "%s: decode q_lens[%d] = %lld != 1", what, i, q);
    if (ctx < 0) return fail(STAGE_ERR_INVALID_ARG, "%s: ctx_lens[%d] < 0", what, i);
    if (ctx + q > cap)
      return fail(STAGE_ERR_CAPACITY, "%s: sequence %d needs %lld tokens > table capacity %lld",
                  what, i, ctx + q, cap);
    if (ctx + q > c.max_position)
      return fail(STAGE_ERR_CAPACITY, "%s: sequence %d reaches position %lld >= max_position %d",
                  what, i, ctx + q - 1, c.max_position);
    *tokens += q;
  }
  return STAGE_OK;
}

stage_status check_step(const stage_model_config& c, int32_t max_tokens, int32_t max_seqs,
                        const stage_batch* pf, const stage_batch* dc, long long* T) {
  long long tp = 0, td = 0;
  stage_status s = check_batch(c, pf, false, "prefill", &tp);
  if (s != STAGE_OK) return s;
  s = check_batch(c, dc, true, "decode", &td);
  if (s != STAGE_OK) return s;
  const long long ns = (pf ? pf->num_seqs : 0) + (dc ? dc->num_seqs : 0);
  if (tp + td > max_tokens)
    return fail(STAGE_ERR_CAPACITY, "step has %lld tokens > max_tokens %d", tp + td, max_tokens);
  if (ns > max_seqs)
    return fail(STAGE_ERR_CAPACITY, "step has %lld sequences > max_seqs %d", ns, max_seqs);
  *T = tp + td;
  return STAGE_OK;
}

stage_status hip_fail(const char* what, hipError_t e) {
  return fail(STAGE_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

void plan_workspace(stage* st) {
  const auto& c = st->cfg;
  const size_t T = st->max_tokens, H = c.hidden, D = c.head_dim;
  const size_t qw = (size_t)c.n_q_heads * D, qkvw = (size_t)(c.n_q_heads + 2 * c.n_kv_heads) * D;
  const size_t F = c.ffn, es = st->esize;
  // GEMM inputs (packed activations) are read in whole 256- or 192-row tiles
  const size_t Tp = std::max((T + 255) / 256 * 256, (T + 191) / 192 * 192);
  const size_t R = st->skinny_rows;
  size_t off = 0;
  auto take = [&](Region& r, size_t bytes) {
    r.off = off;
    r.bytes = bytes;
    off = align_up(off + bytes, 256);
  };
  take(st->r_x, T * H * 4);
  take(st->r_h, Tp * H * es);
  // split-K planes of small tiled steps (bf16)
  const bool mid = c.dtype == STAGE_BF16 && T > R;
  take(st->r_qkv, std::max({T * qkvw, (size_t)st->s_qkv * R * qkvw,
                            mid ? mid_capacity((int)T, (int)qkvw) : 0}) * 4);
  take(st->r_kvpart, c.dtype == STAGE_BF16 ? kMaxKvSplits * T * (qkvw - qw) * 4 : 0);
  take(st->r_q, T * qw * es);
  take(st->r_attn, Tp * qw * es);
  take(st->r_m, Tp * F * es);
  const size_t gu_rows = c.dtype == STAGE_F32 ? T : (st->s_gu > 1 ? (size_t)st->s_gu * R : 0);
  take(st->r_gu, gu_rows * 2 * F * 4);
  // split-K planes of the O / down products of skinny steps and of the last
  // rows of a large step, the mid-split planes, and the QKV planes of the
  // last rows (only one of them is live at a time)
  take(st->r_part_x, std::max({(size_t)std::max(st->s_o, st->s_down) * R * H,
                               mid ? mid_capacity((int)T, (int)H) : 0,
                               mid ? (size_t)st->s_qkv * R * qkvw : 0}) *
                         4);
  const size_t max_items = st->max_ditems;
  take(st->r_part_o, max_items * qw * 4);
  take(st->r_part_ml, max_items * c.n_q_heads * 2 * 4);
  // metadata: tok_seq, tok_pos [T]; decode items [max_items][4];
  // item_start [max_seqs + 1]; tok_rows [max_seqs]; prefill items [T + max_seqs][4];
  // decode item dispatch order [max_items]
  st->meta_ints = 2 * T + 4 * max_items + 2 * (size_t)st->max_seqs + 1 +
                  4 * (T + (size_t)st->max_seqs) + max_items;
  take(st->r_meta, st->meta_ints * 4);
  take(st->r_cos, (size_t)c.max_position * (D / 2) * 4);
  take(st->r_sin, (size_t)c.max_position * (D / 2) * 4);
  st->ws_bytes = off;
}

struct StepMeta {
  int32_t *tok_seq, *tok_pos;
  DecodeItem* ditems;
  int32_t *item_start, *tok_rows;
  int32_t* ditem_order;  // decode items in dispatch order (longest key range first)
  PrefillItem* pitems;
  int n_ditems = 0, n_pitems = 0;
};

// Lay out the metadata arrays over a base pointer (host staging or device).
StepMeta meta_view(const stage* st, int32_t* base) {
  const size_t T = st->max_tokens;
  const size_t max_items = st->max_ditems;
  StepMeta m;
  m.tok_seq = base;
  m.tok_pos = base + T;
  m.ditems = reinterpret_cast<DecodeItem*>(base + 2 * T);
  m.item_start = base + 2 * T + 4 * max_items;
  m.tok_rows = m.item_start + st->max_seqs + 1;
  m.pitems = reinterpret_cast<PrefillItem*>(m.tok_rows + st->max_seqs);
  m.ditem_order = reinterpret_cast<int32_t*>(m.pitems + T + st->max_seqs);
  return m;
}

// Fill the step metadata. Returns false (having written nothing past the
// item capacity) if the decode split plan would exceed max_ditems, which the
// bound of max_decode_items rules out.
bool build_meta(const stage* st, const stage_batch* pf, const stage_batch* dc, StepMeta& m) {
  const int np = pf ? pf->num_seqs : 0, nd = dc ? dc->num_seqs : 0;
  int row = 0;
  const int ppw = prefill_item_positions((DType)st->cfg.dtype,
                                         st->cfg.n_q_heads / st->cfg.n_kv_heads);
  m.n_pitems = 0;
  for (int s = 0; s < np; ++s) {
    const int q = pf->q_lens[s], ctx = pf->ctx_lens[s];
    for (int i = 0; i < q; ++i) {
      m.tok_seq[row + i] = s;
      m.tok_pos[row + i] = ctx + i;
    }
    for (int off = 0; off < q; off += ppw)
      m.pitems[m.n_pitems++] = PrefillItem{s, row + off, ctx + off, std::min(ppw, q - off)};
    row += q;
  }
  // Longest key ranges first, so the slowest waves start first.
  std::stable_sort(m.pitems, m.pitems + m.n_pitems, [](const PrefillItem& a, const PrefillItem& b) {
    return a.p0 + a.npos > b.p0 + b.npos;
  });
  m.n_ditems = 0;
  // Key blocks per decode split: enough splits that the batch launches about
  // `attn_waves` waves (one round on the chip), at least kSplitMinBlocks
  // blocks each, at most kMaxSplits splits per sequence.
  long long units = 0;
  for (int j = 0; j < nd; ++j) units += (dc->ctx_lens[j] + kBlock) / kBlock;
  units *= st->cfg.n_kv_heads;
  const int waves = decode_waves(st->attn_waves, nd, st->attn_scale);
  const int bps_target = (int)std::max<long long>(kSplitMinBlocks, (units + waves - 1) / waves);
  for (int j = 0; j < nd; ++j) {
    const int ctx = dc->ctx_lens[j];
    const int g = np + j;
    m.tok_seq[row] = g;
    m.tok_pos[row] = ctx;
    m.tok_rows[j] = row;
    m.item_start[j] = m.n_ditems;
    ++row;
    if (st->cfg.dtype != STAGE_BF16) continue;  // fp32 attention needs no split plan
    const int keys = ctx + 1;
    const int nb = (keys + kBlock - 1) / kBlock;
    int splits = std::min(kMaxSplits, std::max(1, (nb + bps_target - 1) / bps_target));
    const int bps = (nb + splits - 1) / splits;
    splits = (nb + bps - 1) / bps;
    if ((size_t)(m.n_ditems + splits) > st->max_ditems) return false;
    for (int sp = 0; sp < splits; ++sp) {
      const int k0 = sp * bps * kBlock;
      const int k1 = std::min(keys, (sp + 1) * bps * kBlock);
      m.ditems[m.n_ditems++] = DecodeItem{row - 1, g, k0, k1};
    }
  }
  m.item_start[nd] = m.n_ditems;
  // Dispatch the longest key ranges first (the splits of one sequence
  // differ by at most one block, those of different sequences by up to 2x),
  // so that the short ones fill the tail of the launch.
  for (int i = 0; i < m.n_ditems; ++i) m.ditem_order[i] = i;
  std::stable_sort(m.ditem_order, m.ditem_order + m.n_ditems, [&](int32_t a, int32_t b) {
    return m.ditems[a].k1 - m.ditems[a].k0 > m.ditems[b].k1 - m.ditems[b].k0;
  });
  return true;
}

hipEvent_t take_event(stage* st) {
  if (!st->free_events.empty()) {
    hipEvent_t e = st->free_events.back();
    st->free_events.pop_back();
    return e;
  }
  // Timing-only events: no system-scope release or acquire when they are
  // recorded (only their timestamps are read, after hipEventSynchronize), so
  // that the op timing does not add an L2 writeback and invalidation around
  // every timed launch.
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

// K splits for the key/value columns of a tiled (prefill) QKV product, or 0
// to run QKV as one product. With T rows in whole 256-row tiles, when the
// query columns alone fill whole rounds of one 256 x 256 workgroup per CU,
// the 2 n_kv d key/value columns would leave most of the chip idle as 256
// tiles of their own; split over K they fill one round exactly (e.g. Llama
// 70B at 2048 rows: 8 x 32 query tiles, then 8 x 8 key/value tiles x 4
// splits).
int qkv_kv_splits(const stage* st, int T) {
  const auto& c = st->cfg;
  const int qw = c.n_q_heads * c.head_dim, kvw = 2 * c.n_kv_heads * c.head_dim;
  if (c.dtype != STAGE_BF16 || T % 256 != 0 || qw % 256 != 0 || kvw % 256 != 0) return 0;
  const long mb = T / 256;
  if ((mb * (qw / 256)) % st->cus != 0) return 0;
  for (int sp = 2; sp <= kMaxKvSplits; sp *= 2)
    if (mb * (kvw / 256) * sp == st->cus && c.hidden % (64 * sp) == 0) return sp;
  return 0;
}

// K splits for an [T, N] x [N, K]^T product of a bf16 tiled step (more rows
// than the split-K decode GEMMs take), or 0. When its 256 x 256 tiles would
// occupy less than half of the CUs for the whole K (e.g. O and down with 32
// tiles per 256 rows), it runs over K ranges into fp32 partial planes that
// the consumer sums (as in decode steps): as many ranges (a power of two, at
// most 8) as keep the launch within one round and the planes within
// kMidRows rows.
int mid_splits(const stage* st, int T, int N, int K) {
  if (st->cfg.dtype != STAGE_BF16 || T <= st->skinny_rows || N % 256 != 0) return 0;
  const int tiles = (T + 255) / 256 * (N / 256);
  if (2 * tiles >= st->cus) return 0;
  int best = 0;
  for (int sp = 2; sp <= kMaxMidSplits; sp *= 2)
    if (tiles * sp <= st->cus && K % (64 * sp) == 0 &&
        (size_t)sp * T * N <= mid_capacity(st->max_tokens, N))
      best = sp;
  return best;
}

// Rows of a large bf16 step past its last multiple of 256 (at most the
// skinny limit of them): the candidates for the split-K skinny kernels
// (row_tail_for), with the rows before them on whole tiles. Only when the
// whole-tile part needs no K splits of its own.
int row_tail(const stage* st, int T) {
  if (st->cfg.dtype != STAGE_BF16 || T <= st->skinny_rows || !st->row_tail_on) return 0;
  const int rt = T % 256, T0 = T - rt;
  if (rt == 0 || rt > st->skinny_rows || T0 < 256) return 0;
  const auto& c = st->cfg;
  const int qw = c.n_q_heads * c.head_dim, qkvw = (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  if (mid_splits(st, T0, qkvw, c.hidden) || mid_splits(st, T0, c.hidden, qw) ||
      mid_splits(st, T0, c.hidden, c.ffn))
    return 0;
  return rt;
}

// Whether a product with N tile columns (N of them in 256-wide tiles; for
// QKV with split key/value columns, the query columns) runs its last rt rows
// on the skinny kernel: only when those rows' extra 256-row tiles would add
// a round of workgroups (a mostly idle one: the product then costs about one
// more round of tiles, against one HBM-bound pass over its weights).
bool row_tail_for(const stage* st, int T, int rt, int N) {
  if (rt == 0 || N % 256 != 0) return false;
  const long cols = N / 256;
  const long with = (T + 255) / 256 * cols, without = (T - rt) / 256 * cols;
  return (with + st->cus - 1) / st->cus > (without + st->cus - 1) / st->cus;
}

// Take the next pinned staging slot of the ring, waiting until the upload
// that last used it has been consumed.
stage_status take_slot(stage* st, int* slot) {
  const int sl = st->ring;
  st->ring = (st->ring + 1) % kRing;
  if (st->staging_used[sl]) {
    hipError_t e = hipEventSynchronize(st->staging_ev[sl]);
    if (e != hipSuccess) return hip_fail("staging event", e);
  }
  *slot = sl;
  return STAGE_OK;
}

// Upload `ints` int32 values from staging slot `slot` to the workspace
// metadata region, in stream order.
stage_status upload_slot(stage* st, int slot, size_t ints, hipStream_t s) {
  hipError_t e = hipMemcpyAsync(st->ws + st->r_meta.off, st->staging[slot], ints * 4,
                                hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return hip_fail("metadata upload", e);
  e = hipEventRecord(st->staging_ev[slot], s);
  if (e != hipSuccess) return hip_fail("metadata event", e);
  st->staging_used[slot] = true;
  return STAGE_OK;
}

// Launch helper: brackets a launch with timing events when enabled.
struct Launcher {
  stage* st;
  hipStream_t s;
  hipError_t err = hipSuccess;
  template <typename F>
  void operator()(int op, F&& f) {
    if (err != hipSuccess) return;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (st->timing) {
      e0 = take_event(st);
      e1 = take_event(st);
      if (!e0 || !e1) {
        err = hipErrorOutOfMemory;
        return;
      }
      if ((err = hipEventRecord(e0, s)) != hipSuccess) return;
    }
    err = f();
    if (err == hipSuccess && st->timing) {
      err = hipEventRecord(e1, s);
      st->pending.push_back(PendingTiming{op, e0, e1});
    }
  }
};

// Debug mode: bring the table rows a batch reads to the host (after the
// stream's earlier work, which may have written them) and check every block
// id the call would read.
stage_status check_tables_on_host(const stage* st, const stage_batch* b, const char* what,
                                  hipStream_t s) {
  if (!b || b->num_seqs == 0) return STAGE_OK;
  std::vector<int32_t> tab((size_t)b->num_seqs * b->max_blocks_per_seq);
  hipError_t e = hipMemcpyAsync(tab.data(), b->block_tables, tab.size() * 4,
                                hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail("block table copy", e);
  for (int i = 0; i < b->num_seqs; ++i) {
    const long long nb = ((long long)b->ctx_lens[i] + b->q_lens[i] + kBlock - 1) / kBlock;
    for (long long j = 0; j < nb; ++j) {
      const int32_t id = tab[(size_t)i * b->max_blocks_per_seq + j];
      if (id < 0 || id >= st->num_blocks)
        return fail(STAGE_ERR_INVALID_ARG, "%s: block_tables[%d][%lld] = %d outside [0, %d)",
                    what, i, j, id, st->num_blocks);
    }
  }
  return STAGE_OK;
}

stage_status run_step(stage* st, const stage_batch* pf, const stage_batch* dc, const void* hin,
                      void* hout, void* stream_v) {
  const auto& c = st->cfg;
  if (!st->ws) return fail(STAGE_ERR_INVALID_ARG, "no workspace bound (stage_bind_workspace)");
  long long T64 = 0;
  stage_status vs = check_step(c, st->max_tokens, st->max_seqs, pf, dc, &T64);
  if (vs != STAGE_OK) return vs;
  const int T = (int)T64;
  if (T == 0) return STAGE_OK;
  if (!hin || !hout) return fail(STAGE_ERR_INVALID_ARG, "hidden_in/hidden_out is NULL");
  hipStream_t s = (hipStream_t)stream_v;
  hipError_t e = hipSetDevice(st->device);
  if (e != hipSuccess) return hip_fail("hipSetDevice", e);
  if (st->check_tables) {
    if ((vs = check_tables_on_host(st, pf, "prefill", s)) != STAGE_OK) return vs;
    if ((vs = check_tables_on_host(st, dc, "decode", s)) != STAGE_OK) return vs;
  }

  const int np = pf ? pf->num_seqs : 0, nd = dc ? dc->num_seqs : 0;
  const DType dt = (DType)c.dtype;
  const bool skinny = dt == DT_BF16 && T <= st->skinny_rows;

  // metadata: host build in a pinned staging slot, one async upload
  int slot = 0;
  if ((vs = take_slot(st, &slot)) != STAGE_OK) return vs;
  StepMeta hm = meta_view(st, st->staging[slot]);
  if (!build_meta(st, pf, dc, hm))
    return fail(STAGE_ERR_CAPACITY, "decode split plan exceeds %zu items", st->max_ditems);
  if ((vs = upload_slot(st, slot, st->meta_ints, s)) != STAGE_OK) return vs;
  StepMeta dm = meta_view(st, st->at<int32_t>(st->r_meta));

  const int H = c.hidden, D = c.head_dim, nq = c.n_q_heads, nkv = c.n_kv_heads, F = c.ffn;
  const int qw = nq * D, qkvw = (nq + 2 * nkv) * D;
  const int Tp = T - nd;
  SegTables tabs{pf && np ? pf->block_tables : nullptr, pf && np ? pf->max_blocks_per_seq : 0, np,
                 dc && nd ? dc->block_tables : nullptr, dc && nd ? dc->max_blocks_per_seq : 0};

  float* x = st->at<float>(st->r_x);
  void* h = st->ws + st->r_h.off;
  float* qkv = st->at<float>(st->r_qkv);
  void* q = st->ws + st->r_q.off;
  void* attn = st->ws + st->r_attn.off;
  void* m = st->ws + st->r_m.off;
  float* gu = st->at<float>(st->r_gu);
  float* part_x = st->at<float>(st->r_part_x);
  const float* cos_t = st->at<float>(st->r_cos);
  const float* sin_t = st->at<float>(st->r_sin);

  // The layer loop on stream ls. Split-K steps leave the O / down
  // projections as partial sums in part_x; the next RMSNorm (or the output
  // cast) adds them to the residual stream. The first layer's input norm
  // (which reads hidden_in) is launched before it.
  // rows [T0, T) of a large step may run on the skinny kernels (row_tail):
  // for each of QKV, O and down separately (rq, ro, rd: 0 or rt)
  const int rt = skinny ? 0 : row_tail(st, T), T0 = T - rt;
  const int kv_splits0 = rt ? qkv_kv_splits(st, T0) : 0;
  const int rq = row_tail_for(st, T, rt, kv_splits0 ? qw : qkvw) ? rt : 0;
  const int ro = row_tail_for(st, T, rt, H) ? rt : 0, rd = ro;
  const int Tq = T - rq, To = T - ro, Td = T - rd;  // rows of each product on tiles
  const int kv_splits = skinny ? 0 : qkv_kv_splits(st, Tq);
  // with split key/value columns the query product applies RoPE (after the
  // q RMSNorm of q/k-norm models) in its epilogue (one 128-column head per
  // wave)
  const bool q_fused = kv_splits > 0 && (!c.qk_norm || st->q_norm_fused) && D == 128 &&
                       nq % 4 == 0 &&
                       st->q_rope_fused;
  const int mq = rt ? 0 : mid_splits(st, T, qkvw, H), mo = rt ? 0 : mid_splits(st, T, H, qw),
            md = rt ? 0 : mid_splits(st, T, H, F);
  // the tail rows of the packed activations (whole 16-row fragments)
  auto tail_rows = [&](const void* act, int K) -> const void* {
    return (const uint16_t*)act + (size_t)(T0 / 16) * (K / 32) * 512;
  };
  auto layers = [&](Launcher& L, hipStream_t ls) {
    Partials pending{nullptr, 0};
    for (int li = 0; li < st->n_layers; ++li) {
      const stage_layer_weights& w = st->layers[li];
      KVLayer kvl{st->kv_pool + (size_t)li * st->kv_layer_bytes, nkv, D};
      if (li > 0)
        L(STAGE_OP_NORM, [&] { return rmsnorm(dt, x, pending, h, w.attn_norm, T, H, c.rms_eps, ls); });

      // where RoPE finds the projection: [T][qkvw], possibly in split planes,
      // or the query columns [T][qw] and split planes of the key/value columns
      ProjSrc qsrc{qkv, qkvw, 1, 0}, kvsrc{qkv + qw, qkvw, 1, 0};
      ProjSrc qtail = qsrc, kvtail = kvsrc;
      if (rq > 0) {
        const size_t plane = (size_t)rq * qkvw;
        qtail = ProjSrc{part_x, qkvw, st->s_qkv, plane};
        kvtail = ProjSrc{part_x + qw, qkvw, st->s_qkv, plane};
        L(STAGE_OP_QKV, [&] {
          return gemm_skinny(tail_rows(h, H), w.w_qkv, rq, qkvw, H, st->s_qkv, false, part_x, ls);
        });
      }
      if (skinny) {
        const size_t plane = (size_t)T * qkvw;
        qsrc = ProjSrc{qkv, qkvw, st->s_qkv, plane};
        kvsrc = ProjSrc{qkv + qw, qkvw, st->s_qkv, plane};
        L(STAGE_OP_QKV, [&] { return gemm_skinny(h, w.w_qkv, T, qkvw, H, st->s_qkv, false, qkv, ls); });
      } else if (mq > 0) {
        const size_t plane = (size_t)T * qkvw;
        qsrc = ProjSrc{qkv, qkvw, mq, plane};
        kvsrc = ProjSrc{qkv + qw, qkvw, mq, plane};
        L(STAGE_OP_QKV, [&] { return gemm_split_k(h, w.w_qkv, T, qkvw, H, mq, qkv, ls); });
      } else if (kv_splits > 0) {
        float* kvpart = st->at<float>(st->r_kvpart);
        const int kvw = qkvw - qw;
        qsrc = ProjSrc{qkv, qw, 1, 0};
        kvsrc = ProjSrc{kvpart, kvw, kv_splits, (size_t)Tq * kvw};
        if (q_fused)
          L(STAGE_OP_QKV, [&] {
            return gemm(dt, EPI_ROPE_Q, h, w.w_qkv, Tq, qw, H, q, ls,
                        RopeRows{dm.tok_pos, cos_t, sin_t, c.qk_norm ? w.q_norm : nullptr,
                                 c.qk_rms_eps});
          });
        else
          L(STAGE_OP_QKV, [&] { return gemm(dt, EPI_STORE_F32, h, w.w_qkv, Tq, qw, H, qkv, ls); });
        L(STAGE_OP_QKV, [&] {
          return gemm_split_k(h, (const uint16_t*)w.w_qkv + (size_t)qw * H, Tq, kvw, H, kv_splits,
                              kvpart, ls);
        });
      } else {
        L(STAGE_OP_QKV, [&] { return gemm(dt, EPI_STORE_F32, h, w.w_qkv, Tq, qkvw, H, qkv, ls); });
      }
      L(STAGE_OP_ROPE_KV, [&] {
        return rope_kv_write(dt, qsrc, kvsrc, qtail, kvtail, Tq, q_fused, q, kvl, dm.tok_seq,
                             dm.tok_pos, tabs, cos_t, sin_t, c.qk_norm ? w.q_norm : nullptr,
                             c.qk_norm ? w.k_norm : nullptr, c.qk_rms_eps, T, nq, ls);
      });

      if (dt == DT_F32) {
        L(STAGE_OP_ATTN, [&] {
          return attn_f32((const float*)q, kvl, tabs, dm.tok_seq, dm.tok_pos, 0, T, nq,
                          (float*)attn, ls);
        });
      } else {
        if (Tp > 0)
          L(STAGE_OP_ATTN, [&] {
            return attn_prefill(dt, q, kvl, tabs, dm.pitems, hm.n_pitems, nq, attn, ls);
          });
        if (nd > 0) {
          L(STAGE_OP_ATTN, [&] {
            return attn_decode(dt, q, kvl, tabs, dm.ditems, dm.ditem_order, hm.n_ditems, nq,
                               st->at<float>(st->r_part_o), st->at<float>(st->r_part_ml), ls);
          });
          L(STAGE_OP_ATTN, [&] {
            return attn_merge(dt, st->at<float>(st->r_part_o), st->at<float>(st->r_part_ml),
                              dm.item_start, dm.tok_rows, nd, nq, nkv, D, attn, ls);
          });
        }
      }

      if (skinny) {
        L(STAGE_OP_O, [&] { return gemm_skinny(attn, w.w_o, T, H, qw, st->s_o, false, part_x, ls); });
        pending = Partials{part_x, st->s_o};
      } else if (mo > 0) {
        L(STAGE_OP_O, [&] { return gemm_split_k(attn, w.w_o, T, H, qw, mo, part_x, ls); });
        pending = Partials{part_x, mo};
      } else {
        L(STAGE_OP_O, [&] { return gemm(dt, EPI_RESID_ADD, attn, w.w_o, To, H, qw, x, ls); });
        if (ro > 0) {
          L(STAGE_OP_O, [&] {
            return gemm_skinny(tail_rows(attn, qw), w.w_o, ro, H, qw, st->s_o, false, part_x, ls);
          });
          pending = Partials{part_x, st->s_o, To};
        }
      }

      L(STAGE_OP_NORM, [&] { return rmsnorm(dt, x, pending, h, w.ffn_norm, T, H, c.rms_eps, ls); });
      pending = Partials{nullptr, 0};

      if (skinny) {
        if (st->s_gu == 1) {
          L(STAGE_OP_GATE_UP, [&] { return gemm_skinny(h, w.w_gate_up, T, 2 * F, H, 1, true, m, ls); });
        } else {
          L(STAGE_OP_GATE_UP, [&] {
            return gemm_skinny(h, w.w_gate_up, T, 2 * F, H, st->s_gu, false, gu, ls);
          });
          L(STAGE_OP_NORM, [&] {
            return swiglu_reduce_bf16(Partials{gu, st->s_gu}, (uint16_t*)m, T, F, ls);
          });
        }
        L(STAGE_OP_DOWN, [&] { return gemm_skinny(m, w.w_down, T, H, F, st->s_down, false, part_x, ls); });
        pending = Partials{part_x, st->s_down};
      } else if (dt == DT_BF16) {
        L(STAGE_OP_GATE_UP, [&] { return gemm(dt, EPI_SWIGLU, h, w.w_gate_up, T, 2 * F, H, m, ls); });
        if (md > 0) {
          L(STAGE_OP_DOWN, [&] { return gemm_split_k(m, w.w_down, T, H, F, md, part_x, ls); });
          pending = Partials{part_x, md};
        } else {
          L(STAGE_OP_DOWN, [&] { return gemm(dt, EPI_RESID_ADD, m, w.w_down, Td, H, F, x, ls); });
          if (rd > 0) {
            L(STAGE_OP_DOWN, [&] {
              return gemm_skinny(tail_rows(m, F), w.w_down, rd, H, F, st->s_down, false, part_x,
                                 ls);
            });
            pending = Partials{part_x, st->s_down, Td};
          }
        }
      } else {
        L(STAGE_OP_GATE_UP, [&] { return gemm(dt, EPI_STORE_F32, h, w.w_gate_up, T, 2 * F, H, gu, ls); });
        L(STAGE_OP_NORM, [&] { return swiglu_f32(gu, (float*)m, T, F, ls); });
        L(STAGE_OP_DOWN, [&] { return gemm(dt, EPI_RESID_ADD, m, w.w_down, T, H, F, x, ls); });
      }
    }
  };
  // what the last layer leaves for the output cast
  const Partials tail = skinny   ? Partials{part_x, st->s_down}
                        : md > 0 ? Partials{part_x, md}
                        : rd > 0 ? Partials{part_x, st->s_down, Td}
                                 : Partials{nullptr, 0};

  Launcher L{st, s};
  L(STAGE_OP_NORM, [&] {
    return embed_norm(dt, hin, x, h, st->layers[0].attn_norm, T, H, c.rms_eps, s);
  });
  layers(L, s);
  L(STAGE_OP_NORM, [&] { return output_cast(dt, x, tail, hout, T, H, s); });

  if (L.err != hipSuccess) return hip_fail("kernel launch", L.err);
  return STAGE_OK;
}

}  // namespace

extern "C" {

stage_status stage_create(const stage_model_config* cfg, int32_t layer_begin, int32_t layer_end,
                          const stage_layer_weights* layers, void* kv_pool, int32_t num_blocks,
                          int32_t max_tokens, int32_t max_seqs, stage_t** out) {
  if (!out) return fail(STAGE_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  stage_status s = check_config(cfg);
  if (s != STAGE_OK) return s;
  if (layer_begin < 0 || layer_end <= layer_begin)
    return fail(STAGE_ERR_INVALID_ARG, "layer range [%d, %d) is empty or negative", layer_begin,
                layer_end);
  if (!layers) return fail(STAGE_ERR_INVALID_ARG, "layers is NULL");
  if (!kv_pool) return fail(STAGE_ERR_INVALID_ARG, "kv_pool is NULL");
  if (num_blocks <= 0 || max_tokens <= 0 || max_seqs <= 0)
    return fail(STAGE_ERR_INVALID_ARG, "num_blocks, max_tokens and max_seqs must be positive");
  const int n = layer_end - layer_begin;
  for (int i = 0; i < n; ++i) {
    const stage_layer_weights& w = layers[i];
    if (!w.attn_norm || !w.w_qkv || !w.w_o || !w.ffn_norm || !w.w_gate_up || !w.w_down)
      return fail(STAGE_ERR_INVALID_ARG, "layer %d: a weight pointer is NULL", layer_begin + i);
    if (cfg->qk_norm && (!w.q_norm || !w.k_norm))
      return fail(STAGE_ERR_INVALID_ARG, "layer %d: q_norm/k_norm NULL with qk_norm set",
                  layer_begin + i);
  }
  int ndev = 0;
  hipError_t e = hipGetDeviceCount(&ndev);
  if (e != hipSuccess || ndev <= 0)
    return fail(STAGE_ERR_DEVICE, "no HIP device available (%s)",
                e != hipSuccess ? hipGetErrorString(e) : "0 devices");
  stage* st = new (std::nothrow) stage();
  if (!st) return fail(STAGE_ERR_OUT_OF_MEMORY, "host allocation failed");
  st->cfg = *cfg;
  st->layer_begin = layer_begin;
  st->n_layers = n;
  st->layers.assign(layers, layers + n);
  st->kv_pool = (char*)kv_pool;
  st->num_blocks = num_blocks;
  st->max_tokens = max_tokens;
  st->max_seqs = max_seqs;
  st->esize = cfg->dtype == STAGE_BF16 ? 2 : 4;
  st->kv_layer_bytes = (size_t)num_blocks * cfg->n_kv_heads * 2 * kBlock * cfg->head_dim * st->esize;
  st->skinny_rows = cfg->dtype == STAGE_BF16 ? std::min(kSkinnyMaxRows, max_tokens) : 0;
  if ((e = hipGetDevice(&st->device)) != hipSuccess) {
    delete st;
    return hip_fail("hipGetDevice", e);
  }
  {
    // Split-K GEMM blocks stream at a roughly fixed rate per CU, so each
    // GEMM gets as many K splits as fill ~90% of the CUs with one block
    // each (more blocks than CUs double up on some CUs and stretch the tail).
    int cus = 256;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, st->device) !=
            hipSuccess ||
        cus <= 0)
      cus = 256;
    st->cus = cus;
    const int blocks = std::max(1, env_int("STAGE_SKINNY_BLOCKS", cus * 9 / 10));
    const int H = cfg->hidden, F = cfg->ffn, qw = cfg->n_q_heads * cfg->head_dim;
    const int qkvw = (cfg->n_q_heads + 2 * cfg->n_kv_heads) * cfg->head_dim;
    // products the k-part kernel takes (K % 128 == 0) are planned for it:
    // one block per CU
    const int kp_blocks = std::max(1, env_int("STAGE_SKINNY_KP_BLOCKS", cus));
    auto splits_for = [&](int N, int K, int max_splits) {
      return skinny_kp_enabled() && K % 128 == 0 ? skinny_kp_splits(N, K, kp_blocks, max_splits)
                                                 : skinny_splits(N, K, blocks, max_splits);
    };
    st->s_qkv = splits_for(qkvw, H, kSkinnyMaxQkvSplits);
    st->s_o = splits_for(H, qw, kSkinnyMaxSplits);
    st->s_gu = splits_for(2 * F, H, kSkinnyMaxSplits);
    st->s_down = splits_for(H, F, kSkinnyMaxSplits);
    st->attn_waves = std::max(64, env_int("STAGE_ATTN_WAVES", 1600));
    st->attn_scale = env_int("STAGE_ATTN_SCALE", 1) != 0;
    st->row_tail_on = env_int("STAGE_ROW_TAIL", 1) != 0;
    st->q_rope_fused = env_int("STAGE_Q_ROPE", 1) != 0;
    st->q_norm_fused = env_int("STAGE_Q_NORM_EPI", 1) != 0;
    st->check_tables = env_int("STAGE_DEBUG", 0) != 0;
  }
  st->max_ditems = cfg->dtype == STAGE_BF16
                       ? max_decode_items(max_seqs,
                                          decode_waves(st->attn_waves, max_seqs, st->attn_scale),
                                          cfg->n_kv_heads)
                       : 0;
  st->uid = g_stage_uid.fetch_add(1) + 1;
  plan_workspace(st);
  {
    const int half = cfg->head_dim / 2;
    const size_t n = (size_t)cfg->max_position * half;
    try {
      st->rope_host.resize(2 * n);
    } catch (const std::bad_alloc&) {
      delete st;
      return fail(STAGE_ERR_OUT_OF_MEMORY, "host allocation of the rotary table failed");
    }
    for (int j = 0; j < half; ++j) {
      const double w = std::pow(cfg->rope_theta, -2.0 * j / cfg->head_dim);
      for (int p = 0; p < cfg->max_position; ++p) {
        const double a = (double)p * w;
        st->rope_host[(size_t)p * half + j] = (float)std::cos(a);
        st->rope_host[n + (size_t)p * half + j] = (float)std::sin(a);
      }
    }
  }
  for (int i = 0; i < kRing; ++i) {
    void* p = nullptr;
    if ((e = hipHostMalloc(&p, st->meta_ints * 4, hipHostMallocDefault)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&st->staging_ev[i], hipEventDisableTiming)) != hipSuccess) {
      if (p) (void)hipHostFree(p);
      stage_destroy(st);
      return hip_fail("pinned staging", e);
    }
    st->staging[i] = (int32_t*)p;
  }
  *out = st;
  return STAGE_OK;
}

size_t stage_workspace_bytes(const stage_t* st) { return st ? st->ws_bytes : 0; }

stage_status stage_bind_workspace(stage_t* st, void* dev, size_t bytes) {
  if (!st || !dev) return fail(STAGE_ERR_INVALID_ARG, "stage or workspace is NULL");
  if (bytes < st->ws_bytes)
    return fail(STAGE_ERR_CAPACITY, "workspace of %zu bytes < required %zu", bytes, st->ws_bytes);
  if (((uintptr_t)dev) % 256 != 0) return fail(STAGE_ERR_INVALID_ARG, "workspace not 256-byte aligned");
  hipError_t e = hipSetDevice(st->device);
  if (e != hipSuccess) return hip_fail("hipSetDevice", e);
  st->ws = (char*)dev;
  const size_t n = st->rope_host.size() / 2;
  if ((e = hipMemcpy(st->ws + st->r_cos.off, st->rope_host.data(), n * 4,
                     hipMemcpyHostToDevice)) != hipSuccess ||
      (e = hipMemcpy(st->ws + st->r_sin.off, st->rope_host.data() + n, n * 4,
                     hipMemcpyHostToDevice)) != hipSuccess) {
    st->ws = nullptr;
    return hip_fail("workspace init", e);
  }
  return STAGE_OK;
}

stage_status stage_prefill(stage_t* st, const stage_batch* batch, const void* hidden_in,
                           void* hidden_out, void* stream) {
  if (!st) return fail(STAGE_ERR_INVALID_ARG, "stage is NULL");
  if (!batch) return fail(STAGE_ERR_INVALID_ARG, "batch is NULL");
  return run_step(st, batch, nullptr, hidden_in, hidden_out, stream);
}

stage_status stage_decode(stage_t* st, const stage_batch* batch, const void* hidden_in,
                          void* hidden_out, void* stream) {
  if (!st) return fail(STAGE_ERR_INVALID_ARG, "stage is NULL");
  if (!batch) return fail(STAGE_ERR_INVALID_ARG, "batch is NULL");
  return run_step(st, nullptr, batch, hidden_in, hidden_out, stream);
}

stage_status stage_step_mixed(stage_t* st, const stage_batch* prefill, const stage_batch* decode,
                              const void* hidden_in, void* hidden_out, void* stream) {
  if (!st) return fail(STAGE_ERR_INVALID_ARG, "stage is NULL");
  return run_step(st, prefill, decode, hidden_in, hidden_out, stream);
}

stage_status stage_decode_noalloc(stage_t* st, const stage_batch* batch, const void* hidden_in,
                                  void* hidden_out, void* stream) {
  if (!st) return fail(STAGE_ERR_INVALID_ARG, "stage is NULL");
  if (!batch) return fail(STAGE_ERR_INVALID_ARG, "batch is NULL");
  if (st->ws_bytes > kStaticScratchBytes)
    return fail(STAGE_ERR_CAPACITY,
                "the stage's workspace (%zu bytes) exceeds the static scratch array (%zu bytes): "
                "create the stage with smaller max_tokens / max_seqs / max_position",
                st->ws_bytes, kStaticScratchBytes);
  if (st->device < 0 || st->device >= kMaxStaticDevices)
    return fail(STAGE_ERR_UNSUPPORTED, "device %d has no static scratch slot", st->device);
  // the checks run_step applies, before anything is enqueued here
  long long T = 0;
  stage_status vs = check_step(st->cfg, st->max_tokens, st->max_seqs, nullptr, batch, &T);
  if (vs != STAGE_OK) return vs;
  if (T == 0) return STAGE_OK;
  if (!hidden_in || !hidden_out) return fail(STAGE_ERR_INVALID_ARG, "hidden_in/hidden_out is NULL");
  hipError_t e = hipSetDevice(st->device);
  if (e != hipSuccess) return hip_fail("hipSetDevice", e);
  void* scr = nullptr;
  if ((e = static_scratch(st->device, &scr)) != hipSuccess)
    return hip_fail("static scratch address", e);
  hipStream_t s = (hipStream_t)stream;
  {
    // the rotary table, unless this stage's last call left it there
    std::lock_guard<std::mutex> lock(g_static_mu);
    if (g_static_owner[st->device] != st->uid) {
      g_static_owner[st->device] = 0;
      const size_t n = st->rope_host.size() / 2;
      char* base = (char*)scr;
      if ((e = hipMemcpyAsync(base + st->r_cos.off, st->rope_host.data(), n * 4,
                              hipMemcpyHostToDevice, s)) != hipSuccess ||
          (e = hipMemcpyAsync(base + st->r_sin.off, st->rope_host.data() + n, n * 4,
                              hipMemcpyHostToDevice, s)) != hipSuccess)
        return hip_fail("rotary table upload", e);
      g_static_owner[st->device] = st->uid;
    }
  }
  // the forward pass of stage_decode over the static array; op timing (which
  // may create events) is not applied to these launches
  char* bound = st->ws;
  const bool timing = st->timing;
  st->ws = (char*)scr;
  st->timing = false;
  vs = run_step(st, nullptr, batch, hidden_in, hidden_out, stream);
  st->ws = bound;
  st->timing = timing;
  return vs;
}

stage_status stage_pack_lm_head(const stage_model_config* cfg, int32_t vocab, const void* src,
                                void* dst, void* stream) {
  stage_status v = check_config(cfg);
  if (v != STAGE_OK) return v;
  if (!src || !dst) return fail(STAGE_ERR_INVALID_ARG, "src/dst is NULL");
  if (src == dst) return fail(STAGE_ERR_INVALID_ARG, "packing cannot run in place");
  if (vocab <= 0) return fail(STAGE_ERR_INVALID_ARG, "vocab must be positive");
  if (cfg->dtype == STAGE_BF16 && vocab % 128 != 0)
    return fail(STAGE_ERR_UNSUPPORTED, "vocab %d is not a multiple of 128", vocab);
  hipStream_t s = (hipStream_t)stream;
  const int H = cfg->hidden;
  hipError_t e;
  if (cfg->dtype == STAGE_F32)
    e = hipMemcpyAsync(dst, src, (size_t)vocab * H * 4, hipMemcpyDeviceToDevice, s);
  else
    e = pack_weight(src, dst, vocab, H, 0, s);
  if (e != hipSuccess) return hip_fail("pack_weight", e);
  return STAGE_OK;
}

stage_status stage_lm_head(stage_t* st, const void* final_norm, const void* w_lm, int32_t vocab,
                           const void* hidden, int32_t hidden_rows, const int32_t* rows,
                           int32_t n_rows, float* logits, void* stream) {
  if (!st) return fail(STAGE_ERR_INVALID_ARG, "stage is NULL");
  if (!st->ws) return fail(STAGE_ERR_INVALID_ARG, "no workspace bound (stage_bind_workspace)");
  if (!final_norm || !w_lm || !hidden || !logits)
    return fail(STAGE_ERR_INVALID_ARG, "final_norm/w_lm/hidden/logits is NULL");
  const auto& c = st->cfg;
  if (vocab <= 0 || hidden_rows < 0 || n_rows < 0)
    return fail(STAGE_ERR_INVALID_ARG, "vocab must be positive, row counts >= 0");
  if (c.dtype == STAGE_BF16 && vocab % 128 != 0)
    return fail(STAGE_ERR_UNSUPPORTED, "vocab %d is not a multiple of 128", vocab);
  if (n_rows == 0) return STAGE_OK;
  if (n_rows > st->max_tokens)
    return fail(STAGE_ERR_CAPACITY, "%d rows > max_tokens %d", n_rows, st->max_tokens);
  if (rows) {
    for (int i = 0; i < n_rows; ++i)
      if (rows[i] < 0 || rows[i] >= hidden_rows)
        return fail(STAGE_ERR_INVALID_ARG, "rows[%d] = %d outside [0, %d)", i, rows[i],
                    hidden_rows);
  } else if (n_rows > hidden_rows) {
    return fail(STAGE_ERR_INVALID_ARG, "%d rows > hidden_rows %d", n_rows, hidden_rows);
  }
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = hipSetDevice(st->device);
  if (e != hipSuccess) return hip_fail("hipSetDevice", e);
  const int32_t* rows_dev = nullptr;
  if (rows) {
    int slot = 0;
    stage_status vs = take_slot(st, &slot);
    if (vs != STAGE_OK) return vs;
    std::memcpy(st->staging[slot], rows, (size_t)n_rows * 4);
    if ((vs = upload_slot(st, slot, n_rows, s)) != STAGE_OK) return vs;
    rows_dev = st->at<int32_t>(st->r_meta);
  }
  const DType dt = (DType)c.dtype;
  const int H = c.hidden;
  float* x = st->at<float>(st->r_x);
  void* h = st->ws + st->r_h.off;
  Launcher L{st, s};
  L(STAGE_OP_LM_HEAD, [&] {
    return embed_norm(dt, hidden, x, h, final_norm, n_rows, H, c.rms_eps, s, rows_dev);
  });
  if (dt == DT_BF16 && n_rows <= st->skinny_rows)
    L(STAGE_OP_LM_HEAD, [&] { return gemm_skinny(h, w_lm, n_rows, vocab, H, 1, false, logits, s); });
  else
    L(STAGE_OP_LM_HEAD, [&] { return gemm(dt, EPI_STORE_F32, h, w_lm, n_rows, vocab, H, logits, s); });
  if (L.err != hipSuccess) return hip_fail("kernel launch", L.err);
  return STAGE_OK;
}

stage_status stage_destroy(stage_t* st) {
  if (!st) return STAGE_OK;
  for (int i = 0; i < kRing; ++i) {
    if (st->staging_ev[i]) {
      if (st->staging_used[i]) (void)hipEventSynchronize(st->staging_ev[i]);
      (void)hipEventDestroy(st->staging_ev[i]);
    }
    if (st->staging[i]) (void)hipHostFree(st->staging[i]);
  }
  for (auto& p : st->pending) {
    (void)hipEventSynchronize(p.e1);
    (void)hipEventDestroy(p.e0);
    (void)hipEventDestroy(p.e1);
  }
  for (auto e : st->free_events) (void)hipEventDestroy(e);
  delete st;
  return STAGE_OK;
}

const char* stage_last_error(void) { return g_err.c_str(); }

stage_status stage_validate_step(const stage_model_config* cfg, int32_t max_tokens,
                                 int32_t max_seqs, const stage_batch* prefill,
                                 const stage_batch* decode) {
  stage_status s = check_config(cfg);
  if (s != STAGE_OK) return s;
  long long T = 0;
  return check_step(*cfg, max_tokens, max_seqs, prefill, decode, &T);
}

stage_status stage_pack_weight(const stage_model_config* cfg, stage_weight_kind kind,
                               const void* src, void* dst, void* stream) {
  stage_status v = check_config(cfg);
  if (v != STAGE_OK) return v;
  if (!src || !dst) return fail(STAGE_ERR_INVALID_ARG, "src/dst is NULL");
  if (src == dst) return fail(STAGE_ERR_INVALID_ARG, "packing cannot run in place");
  const int H = cfg->hidden, F = cfg->ffn, qw = cfg->n_q_heads * cfg->head_dim;
  const int qkvw = (cfg->n_q_heads + 2 * cfg->n_kv_heads) * cfg->head_dim;
  int N = 0, K = 0, ffn = 0;
  static_assert(sizeof(stage_weight_kind) == sizeof(int32_t), "stage_weight_kind is 32-bit");
  int32_t kind_raw;
  std::memcpy(&kind_raw, &kind, sizeof kind_raw);
  switch (kind_raw) {
    case STAGE_W_QKV: N = qkvw; K = H; break;
    case STAGE_W_O: N = H; K = qw; break;
    case STAGE_W_GATE_UP: N = 2 * F; K = H; ffn = F; break;
    case STAGE_W_DOWN: N = H; K = F; break;
    default: return fail(STAGE_ERR_INVALID_ARG, "unknown weight kind %d", (int)kind_raw);
  }
  hipStream_t s = (hipStream_t)stream;
  hipError_t e;
  if (cfg->dtype == STAGE_F32)
    e = hipMemcpyAsync(dst, src, (size_t)N * K * 4, hipMemcpyDeviceToDevice, s);
  else
    e = pack_weight(src, dst, N, K, ffn, s);
  if (e != hipSuccess) return hip_fail("pack_weight", e);
  return STAGE_OK;
}

stage_status stage_copy_probe(const void* src, void* dst, size_t bytes, void* stream) {
  if (!src || !dst) return fail(STAGE_ERR_INVALID_ARG, "src/dst is NULL");
  if (bytes % 16 != 0 || (uintptr_t)src % 16 != 0 || (uintptr_t)dst % 16 != 0)
    return fail(STAGE_ERR_INVALID_ARG, "copy probe needs 16-byte aligned pointers and sizes");
  const char* a = (const char*)src;
  const char* b = (const char*)dst;
  if (a < b + bytes && b < a + bytes) return fail(STAGE_ERR_INVALID_ARG, "copy probe buffers overlap");
  hipError_t e = copy_probe(src, dst, bytes, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail("copy_probe", e);
  return STAGE_OK;
}

stage_status stage_set_op_timing(stage_t* st, int32_t enable) {
  if (!st) return fail(STAGE_ERR_INVALID_ARG, "stage is NULL");
  st->timing = enable != 0;
  return STAGE_OK;
}

stage_status stage_read_op_times(stage_t* st, double* ms, int64_t* launches) {
  if (!st || !ms || !launches) return fail(STAGE_ERR_INVALID_ARG, "NULL argument");
  for (auto& p : st->pending) {
    hipError_t e = hipEventSynchronize(p.e1);
    if (e != hipSuccess) return hip_fail("timing event", e);
    float t = 0.f;
    if (hipEventElapsedTime(&t, p.e0, p.e1) == hipSuccess) {
      st->op_ms[p.op] += t;
      st->op_launches[p.op] += 1;
    }
    st->free_events.push_back(p.e0);
    st->free_events.push_back(p.e1);
  }
  st->pending.clear();
  for (int i = 0; i < STAGE_OP_COUNT; ++i) {
    ms[i] = st->op_ms[i];
    launches[i] = st->op_launches[i];
    st->op_ms[i] = 0.0;
    st->op_launches[i] = 0;
  }
  return STAGE_OK;
}

}  // extern "C"
