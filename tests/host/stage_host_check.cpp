// Sanitizer check of the library's host code (test code only).
//
// Built with g++ -fsanitize=address,undefined together with the library's
// host sources (stage.cpp, store.cpp, plan.cpp) against a host-only stand-in
// of the HIP runtime (tests/host/include/hip/hip_runtime.h). "Device"
// memory is host memory here, every HIP copy is a memcpy and every kernel
// launcher is a stub, so the sanitizers see each host-side access the
// runtime makes: argument validation, workspace planning, the step metadata
// that build_meta writes into the pinned staging ring and its upload into
// the workspace, the rotary table, the debug-mode block-table check, op
// timing, the static-scratch entry point and the store calls. The launcher
// stubs also check that the work items a launch would read lie inside the
// workspace. Exit status 0 and a last line "host check passed" on success.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <random>
#include <vector>

#include "../../include/stage.h"
#include "../../paper_2606_18600_amd/csrc/kernels.hpp"

// ---------------------------------------------------------------- HIP stand-in
namespace {
int g_launches = 0;
std::map<const void*, size_t> g_live;  // host allocations standing in for device memory
const char* g_ws = nullptr;            // the workspace of the call in progress
size_t g_ws_bytes = 0;

void fail_check(const char* what) {
  std::fprintf(stderr, "host check failed: %s\n", what);
  std::exit(1);
}
#define CHECK(c)                \
  do {                          \
    if (!(c)) fail_check(#c);   \
  } while (0)

void* dev_alloc(size_t n) {
  void* p = nullptr;
  if (posix_memalign(&p, 256, n ? n : 1) != 0) fail_check("host allocation");
  g_live[p] = n;
  return p;
}
void dev_free(void* p) {
  g_live.erase(p);
  std::free(p);
}
// A pointer range inside one live allocation (the workspace counts as one).
bool inside(const void* p, size_t n) {
  if (g_ws && (const char*)p >= g_ws && (const char*)p + n <= g_ws + g_ws_bytes) return true;
  auto it = g_live.upper_bound(p);
  if (it == g_live.begin()) return false;
  --it;
  return (const char*)p + n <= (const char*)it->first + it->second;
}
struct FakeEvent {
  int id;
};

// What the launches of the current step saw (the metadata lives in host
// memory here, so the stubs can read it back and check it).
int g_T = 0;                      // rows of the step (embed_norm)
const int32_t* g_tok_seq = nullptr;
const int32_t* g_tok_pos = nullptr;
const stage_k::DecodeItem* g_ditems = nullptr;
int g_n_ditems = 0;
}  // namespace

hipError_t hipGetDeviceCount(int* c) { *c = 1; return hipSuccess; }
hipError_t hipGetDevice(int* d) { *d = 0; return hipSuccess; }
hipError_t hipSetDevice(int d) { return d == 0 ? hipSuccess : hipErrorInvalidDevice; }
hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t, int) { *v = 256; return hipSuccess; }
const char* hipGetErrorString(hipError_t) { return "stand-in error"; }
hipError_t hipMalloc(void** p, size_t n) { *p = dev_alloc(n); return hipSuccess; }
hipError_t hipFree(void* p) { dev_free(p); return hipSuccess; }
hipError_t hipHostMalloc(void** p, size_t n, unsigned) { *p = dev_alloc(n); return hipSuccess; }
hipError_t hipHostFree(void* p) { dev_free(p); return hipSuccess; }
hipError_t hipMemset(void* p, int v, size_t n) { std::memset(p, v, n); return hipSuccess; }
hipError_t hipMemcpy(void* d, const void* s, size_t n, hipMemcpyKind) {
  std::memcpy(d, s, n);
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void* d, const void* s, size_t n, hipMemcpyKind, hipStream_t) {
  std::memcpy(d, s, n);
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipEventCreate(hipEvent_t* e) {
  *e = (hipEvent_t) new FakeEvent{0};
  return hipSuccess;
}
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
hipError_t hipEventDestroy(hipEvent_t e) {
  delete (FakeEvent*)e;
  return hipSuccess;
}
hipError_t hipEventElapsedTime(float* ms, hipEvent_t, hipEvent_t) { *ms = 0.001f; return hipSuccess; }
hipError_t hipIpcGetMemHandle(hipIpcMemHandle_t* h, void* p) {
  std::memset(h, 0, sizeof *h);
  std::memcpy(h->reserved, &p, sizeof p);
  return hipSuccess;
}
hipError_t hipIpcOpenMemHandle(void** p, hipIpcMemHandle_t h, unsigned) {
  std::memcpy(p, h.reserved, sizeof *p);
  return hipSuccess;
}
hipError_t hipIpcCloseMemHandle(void*) { return hipSuccess; }

// ----------------------------------------------------------- launcher stubs
namespace stage_k {
hipError_t static_scratch(int device, void** ptr) {
  static void* p = nullptr;
  if (device != 0) return hipErrorInvalidDevice;
  if (!p) p = dev_alloc(kStaticScratchBytes);
  *ptr = p;
  return hipSuccess;
}
hipError_t embed_norm(DType, const void*, float*, void*, const void*, int T, int, float,
                      hipStream_t, const int32_t*) {
  ++g_launches;
  g_T = T;
  return hipSuccess;
}
hipError_t rmsnorm(DType, float*, Partials, void*, const void*, int, int, float, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}
hipError_t output_cast(DType, const float*, Partials, void*, int, int, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}
hipError_t rope_kv_write(DType, ProjSrc, ProjSrc, ProjSrc, ProjSrc, int, bool, void*, KVLayer,
                         const int32_t* tok_seq, const int32_t* tok_pos, SegTables,
                         const float* cos_tab, const float*, const void*, const void*, float,
                         int T, int, hipStream_t) {
  ++g_launches;
  CHECK(T == g_T);
  CHECK(inside(tok_seq, (size_t)T * 4) && inside(tok_pos, (size_t)T * 4));
  CHECK(inside(cos_tab, 4));
  for (int t = 0; t < T; ++t) CHECK(tok_seq[t] >= 0 && tok_pos[t] >= 0);
  g_tok_seq = tok_seq;
  g_tok_pos = tok_pos;
  return hipSuccess;
}
hipError_t swiglu_f32(const float*, float*, int, int, hipStream_t) { ++g_launches; return hipSuccess; }
hipError_t swiglu_reduce_bf16(Partials, uint16_t*, int, int, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}
hipError_t pack_weight(const void*, void*, int, int, int, hipStream_t) { ++g_launches; return hipSuccess; }
hipError_t copy_probe(const void*, void*, size_t, hipStream_t) { ++g_launches; return hipSuccess; }
hipError_t gemm_skinny(const void*, const void*, int M, int N, int K, int splits, bool swiglu, void*,
                       hipStream_t) {
  ++g_launches;
  CHECK(M >= 1 && M <= 128 && N % 64 == 0 && K % 64 == 0 && splits >= 1);
  CHECK(!swiglu || splits == 1);
  const int kb = skinny_kp_used(K, splits, swiglu) ? skinny_kp_kb_len(K, splits)
                                                   : skinny_kb_len(K, splits);
  CHECK((K + kb - 1) / kb == splits);
  return hipSuccess;
}
hipError_t gemm_split_k(const void*, const void*, int M, int N, int K, int splits, float*,
                        hipStream_t) {
  ++g_launches;
  CHECK(M >= 1 && splits >= 1 && N % 256 == 0 && K % (64 * splits) == 0);
  return hipSuccess;
}
hipError_t gemm(DType, Epilogue, const void*, const void*, int M, int N, int K, void*, hipStream_t,
                RopeRows) {
  ++g_launches;
  CHECK(M >= 1 && N >= 1 && K >= 1);
  return hipSuccess;
}
hipError_t attn_decode(DType, const void*, KVLayer, SegTables, const DecodeItem* items,
                       const int32_t* order, int n, int, float*, float*, hipStream_t) {
  ++g_launches;
  CHECK(n >= 1 && inside(items, (size_t)n * sizeof(DecodeItem)));
  // the dispatch order is a permutation of the items, longest key range first
  CHECK(inside(order, (size_t)n * 4));
  std::vector<char> hit(n, 0);
  for (int b = 0; b < n; ++b) {
    CHECK(order[b] >= 0 && order[b] < n && !hit[order[b]]);
    hit[order[b]] = 1;
    if (b > 0)
      CHECK(items[order[b - 1]].k1 - items[order[b - 1]].k0 >=
            items[order[b]].k1 - items[order[b]].k0);
  }
  for (int i = 0; i < n; ++i) {
    const DecodeItem& it = items[i];
    CHECK(it.tok >= 0 && it.tok < g_T);
    CHECK(it.k0 >= 0 && it.k0 < it.k1 && it.k0 % kBlock == 0);
    CHECK(it.k1 <= g_tok_pos[it.tok] + 1);
    CHECK(it.seq == g_tok_seq[it.tok]);
  }
  g_ditems = items;
  g_n_ditems = n;
  return hipSuccess;
}
hipError_t attn_merge(DType, const float*, const float*, const int32_t* starts,
                      const int32_t* rows, int n_tok, int, int, int, void*, hipStream_t) {
  ++g_launches;
  CHECK(inside(starts, (size_t)(n_tok + 1) * 4) && inside(rows, (size_t)n_tok * 4));
  // every decode token's splits: consecutive items covering keys [0, pos]
  CHECK(starts[0] == 0 && starts[n_tok] == g_n_ditems);
  for (int j = 0; j < n_tok; ++j) {
    CHECK(starts[j] < starts[j + 1]);
    const int row = rows[j];
    CHECK(row >= 0 && row < g_T);
    int next = 0;
    for (int i = starts[j]; i < starts[j + 1]; ++i) {
      CHECK(g_ditems[i].tok == row && g_ditems[i].k0 == next);
      next = g_ditems[i].k1;
    }
    CHECK(next == g_tok_pos[row] + 1);
  }
  return hipSuccess;
}
hipError_t attn_prefill(DType, const void*, KVLayer kv, SegTables, const PrefillItem* items,
                        int n, int n_q, void*, hipStream_t) {
  ++g_launches;
  CHECK(n >= 1 && inside(items, (size_t)n * sizeof(PrefillItem)));
  // the items cover the prefill rows [0, covered) exactly once, each within
  // one sequence and at most one work item's positions
  std::vector<char> seen(g_T, 0);
  const int ppw = prefill_item_positions(DT_BF16, n_q / kv.n_kv);
  int covered = 0;
  for (int i = 0; i < n; ++i) {
    const PrefillItem& it = items[i];
    CHECK(it.npos >= 1 && it.npos <= ppw && it.t0 >= 0 && it.t0 + it.npos <= g_T);
    for (int r = it.t0; r < it.t0 + it.npos; ++r) {
      CHECK(!seen[r]);
      seen[r] = 1;
      CHECK(g_tok_seq[r] == it.seq && g_tok_pos[r] == it.p0 + (r - it.t0));
    }
    covered += it.npos;
  }
  for (int r = 0; r < covered; ++r) CHECK(seen[r]);
  return hipSuccess;
}
hipError_t attn_f32(const float*, KVLayer, SegTables, const int32_t* seq, const int32_t* pos, int t0,
                    int n, int, float*, hipStream_t) {
  ++g_launches;
  CHECK(inside(seq + t0, (size_t)n * 4) && inside(pos + t0, (size_t)n * 4));
  return hipSuccess;
}
}  // namespace stage_k

// ---------------------------------------------------------------- scenarios
namespace {

std::mt19937 rng(2606);
int uni(int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); }

stage_model_config config(int hidden, int nq, int nkv, int d, int ffn, int qk, stage_dtype dt,
                          int max_pos = 8192) {
  stage_model_config c{};
  c.hidden = hidden;
  c.n_q_heads = nq;
  c.n_kv_heads = nkv;
  c.head_dim = d;
  c.ffn = ffn;
  c.qk_norm = qk;
  c.block_size = 16;
  c.rms_eps = 1e-5f;
  c.qk_rms_eps = 1e-6f;
  c.rope_theta = 5e5;
  c.max_position = max_pos;
  c.dtype = dt;
  return c;
}

struct Model {
  stage_model_config cfg;
  std::vector<std::vector<void*>> bufs;
  std::vector<stage_layer_weights> layers;
  void* kv = nullptr;
  int num_blocks = 0;
  // Weights and the KV pool are only passed through to the (stub) kernels,
  // so small placeholders stand in for them; gains are real-sized (the LM
  // head passes one on).
  Model(const stage_model_config& c, int n_layers, int nb) : cfg(c), num_blocks(nb) {
    const size_t es = c.dtype == STAGE_BF16 ? 2 : 4;
    for (int l = 0; l < n_layers; ++l) {
      std::vector<void*> b;
      for (int f = 0; f < 8; ++f) b.push_back(dev_alloc((size_t)c.hidden * es));
      layers.push_back({b[0], b[1], b[2], b[3], b[4], b[5], b[6], b[7]});
      bufs.push_back(b);
    }
    kv = dev_alloc(256);
  }
  ~Model() {
    for (auto& b : bufs)
      for (void* p : b) dev_free(p);
    dev_free(kv);
  }
};

// One random step that fits the stage; returns T (0 if nothing was built).
struct Step {
  std::vector<int32_t> pq, pc, dc, ones;
  std::vector<int32_t> pbt, dbt;
  int max_blocks = 0;
};

Step random_step(int max_tokens, int max_seqs, int num_blocks, int max_pos, bool prefill, bool decode) {
  Step s;
  const int max_ctx = std::min(max_pos - 1, 6000);
  s.max_blocks = (max_ctx + 1 + 15) / 16 + 1;
  int budget = max_tokens, seqs = max_seqs;
  if (decode) {
    const int nd = uni(1, std::max(1, std::min(seqs - (prefill ? 1 : 0), 200)));
    for (int i = 0; i < nd && budget > 0; ++i) {
      s.dc.push_back(uni(0, max_ctx - 1));
      s.ones.push_back(1);
      --budget;
      --seqs;
    }
  }
  if (prefill) {
    while (budget > 0 && seqs > 0 && (s.pq.empty() || uni(0, 3) > 0)) {
      const int q = uni(1, std::min(budget, 2500));
      const int c = uni(0, std::max(0, std::min(max_ctx - q, 3000)));
      if (c + q > max_ctx) break;
      s.pq.push_back(q);
      s.pc.push_back(c);
      budget -= q;
      --seqs;
    }
  }
  auto fill = [&](std::vector<int32_t>& bt, size_t n) {
    bt.resize(std::max<size_t>(1, n) * s.max_blocks);
    for (auto& v : bt) v = uni(0, num_blocks - 1);
  };
  fill(s.pbt, s.pq.size());
  fill(s.dbt, s.dc.size());
  return s;
}

void run_shapes() {
  struct Shape {
    int hidden, nq, nkv, d, ffn, qk;
  };
  const Shape shapes[] = {{256, 4, 2, 64, 704, 0},     {512, 8, 1, 128, 768, 1},
                          {256, 4, 4, 64, 512, 0},     {256, 16, 1, 64, 512, 0},
                          {512, 16, 1, 128, 768, 1},   {8192, 64, 8, 128, 28672, 0},
                          {5120, 64, 8, 128, 25600, 1}, {8192, 8, 1, 128, 3584, 0}};
  int calls = 0;
  for (const Shape& sh : shapes) {
    for (stage_dtype dt : {STAGE_BF16, STAGE_F32}) {
      if (sh.hidden >= 5120 && dt == STAGE_F32) continue;
      const int max_tokens = sh.hidden >= 5120 ? 2176 : 1024, max_seqs = sh.hidden >= 5120 ? 160 : 48;
      const int nb = 4096;
      stage_model_config cfg = config(sh.hidden, sh.nq, sh.nkv, sh.d, sh.ffn, sh.qk, dt);
      Model m(cfg, 2, nb);
      for (int debug = 0; debug < 2; ++debug) {
        if (debug) setenv("STAGE_DEBUG", "1", 1);
        stage_t* st = nullptr;
        CHECK(stage_create(&cfg, 3, 5, m.layers.data(), m.kv, nb, max_tokens, max_seqs, &st) == STAGE_OK);
        unsetenv("STAGE_DEBUG");
        const size_t wsb = stage_workspace_bytes(st);
        void* ws = dev_alloc(wsb);
        CHECK(stage_bind_workspace(st, ws, wsb) == STAGE_OK);
        g_ws = (const char*)ws;
        g_ws_bytes = wsb;
        stage_set_op_timing(st, debug);
        const size_t es = dt == STAGE_BF16 ? 2 : 4;
        void* hin = dev_alloc((size_t)max_tokens * sh.hidden * es);
        void* hout = dev_alloc((size_t)max_tokens * sh.hidden * es);
        for (int it = 0; it < 36; ++it) {
          const int kind = it % 3;  // 0 prefill, 1 decode, 2 mixed
          Step s = random_step(max_tokens, max_seqs, nb, cfg.max_position, kind != 1, kind != 0);
          int32_t* pbt = (int32_t*)dev_alloc(s.pbt.size() * 4);
          int32_t* dbt = (int32_t*)dev_alloc(s.dbt.size() * 4);
          std::memcpy(pbt, s.pbt.data(), s.pbt.size() * 4);
          std::memcpy(dbt, s.dbt.data(), s.dbt.size() * 4);
          stage_batch pb{(int32_t)s.pq.size(), s.pq.data(), s.pc.data(), pbt, s.max_blocks};
          stage_batch db{(int32_t)s.dc.size(), s.ones.data(), s.dc.data(), dbt, s.max_blocks};
          stage_status r;
          if (kind == 0) r = stage_prefill(st, &pb, hin, hout, nullptr);
          else if (kind == 1) r = dt == STAGE_BF16 && it % 2 ? stage_decode_noalloc(st, &db, hin, hout, nullptr)
                                                             : stage_decode(st, &db, hin, hout, nullptr);
          else r = stage_step_mixed(st, &pb, &db, hin, hout, nullptr);
          if (r != STAGE_OK && r != STAGE_ERR_CAPACITY) {
            std::fprintf(stderr, "unexpected status %d: %s\n", (int)r, stage_last_error());
            fail_check("forward call");
          }
          ++calls;
          // a table entry outside the pool is caught in debug mode only
          if (debug && !s.dc.empty()) {
            dbt[0] = nb;
            const int before = g_launches;
            CHECK(stage_decode(st, &db, hin, hout, nullptr) == STAGE_ERR_INVALID_ARG);
            CHECK(g_launches == before);
          }
          dev_free(pbt);
          dev_free(dbt);
        }
        // the LM head with a row selection
        {
          const int vocab = 1024;
          void* w = dev_alloc((size_t)vocab * sh.hidden * es);
          float* logits = (float*)dev_alloc((size_t)64 * vocab * 4);
          std::vector<int32_t> rows(64);
          for (auto& r : rows) r = uni(0, max_tokens - 1);
          CHECK(stage_lm_head(st, m.bufs[0][0], w, vocab, hin, max_tokens, rows.data(), 64, logits,
                              nullptr) == STAGE_OK);
          rows[5] = max_tokens;
          CHECK(stage_lm_head(st, m.bufs[0][0], w, vocab, hin, max_tokens, rows.data(), 64, logits,
                              nullptr) == STAGE_ERR_INVALID_ARG);
          dev_free(w);
          dev_free(logits);
        }
        double ms[STAGE_OP_COUNT];
        int64_t n[STAGE_OP_COUNT];
        CHECK(stage_read_op_times(st, ms, n) == STAGE_OK);
        g_ws = nullptr;
        CHECK(stage_destroy(st) == STAGE_OK);
        dev_free(ws);
        dev_free(hin);
        dev_free(hout);
      }
    }
  }
  std::printf("forward calls: %d\n", calls);
}

void run_validation() {
  stage_model_config cfg = config(256, 4, 2, 64, 704, 0, STAGE_BF16, 4096);
  int invalid = 0;
  for (int it = 0; it < 20000; ++it) {
    const int ns = uni(0, 6);
    std::vector<int32_t> q(ns), c(ns);
    for (int i = 0; i < ns; ++i) {
      q[i] = uni(-2, 300);
      c[i] = uni(-2, 5000);
    }
    const int mb = uni(-1, 400);
    stage_batch b{ns, q.data(), c.data(), (const int32_t*)0x1000, mb};
    const int which = uni(0, 2);
    const stage_status r = which == 0 ? stage_validate_step(&cfg, 512, 8, &b, nullptr)
                           : which == 1 ? stage_validate_step(&cfg, 512, 8, nullptr, &b)
                                        : stage_validate_step(&cfg, 512, 8, &b, &b);
    CHECK(r == STAGE_OK || r == STAGE_ERR_INVALID_ARG || r == STAGE_ERR_CAPACITY);
    invalid += r != STAGE_OK;
  }
  // bad configurations
  for (int it = 0; it < 2000; ++it) {
    stage_model_config b = config(uni(-1, 20000), uni(-1, 70), uni(-1, 9), uni(0, 160),
                                  uni(-1, 40000), uni(-1, 2), STAGE_BF16, uni(-1, 100000));
    const int32_t raw_dtype = uni(-1, 2);  // what a C caller may store in the enum field
    std::memcpy(&b.dtype, &raw_dtype, sizeof raw_dtype);
    const stage_status r = stage_validate_step(&b, 64, 4, nullptr, nullptr);
    CHECK(r == STAGE_OK || r == STAGE_ERR_INVALID_ARG || r == STAGE_ERR_UNSUPPORTED);
  }
  std::printf("validation cases: 22000 (%d steps rejected)\n", invalid);
}

void run_store() {
  void* p = nullptr;
  stage_ipc_handle h;
  CHECK(stage_store_alloc(4096, &p, &h) == STAGE_OK && p);
  std::vector<char> src(4096, 7);
  CHECK(stage_store_write(p, src.data(), src.size(), nullptr) == STAGE_OK);
  void* q = nullptr;
  CHECK(stage_store_attach(&h, &q) == STAGE_OK && q == p);
  CHECK(std::memcmp(q, src.data(), src.size()) == 0);
  CHECK(stage_store_detach(q) == STAGE_OK);
  CHECK(stage_store_free(p) == STAGE_OK);
  CHECK(stage_store_alloc((size_t)1 << 31, &p, &h) == STAGE_ERR_CAPACITY);
}

}  // namespace

int main() {
  run_validation();
  run_shapes();
  run_store();
  std::printf("host check passed\n");
  return 0;
}
