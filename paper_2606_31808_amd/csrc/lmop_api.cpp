// Host runtime behind include/lmop.h: argument checks, early deduplication,
// token-budget row batching, the prefix tree with its KV storage, the layer
// loop that drives the gfx950 kernels, the constrained decode loop and
// per-kernel timing.
#include "lmop.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <set>
#include <string>
#include <type_traits>
#include <unordered_map>
#include <vector>

#include "kernels.h"

using namespace lmop;

namespace {

constexpr int kDefaultBatchTokens = 16384;
// a library-allocated own-KV store above this size is released after each call
constexpr size_t kKeepOwnKvBytes = size_t(1) << 30;
// Scratch of lmop_eval_rows_noalloc: a static device array, one per GPU the
// library runs on, held until the process ends
constexpr size_t kNoAllocScratchBytes = size_t(256) << 20;
constexpr int kMaxBatchRows = 2048;
// own-KV bytes of one integer-decode group (also at most half the free memory)
constexpr size_t kDecodeGroupBytes = size_t(24) << 30;
// longest sequence, and largest token budget of one batch; both keep every
// KV store within the attention kernel's kMaxStoreSlots
constexpr int kMaxSeq = 1 << 20;
constexpr int kMaxBatchBudget = 1 << 21;

int round_up(int x, int m) { return (x + m - 1) / m * m; }
int64_t round_up64(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// The scratch of lmop_eval_rows_noalloc.  In host code this name is not a
// device address: each ctx looks up the array's address on its own device
// once (bind_static_scratch) and passes that address to the kernels.
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

struct LayerW {
  float* attn_norm = nullptr;
  float* mlp_norm = nullptr;
  PackedW qkv, o, gu, down;
};

struct Stat {
  int64_t launches = 0;                 // all launches while profiling is on
  int64_t timed = 0;                    // the sampled ones, timed with events
  double ms = 0, flops = 0, bytes = 0;  // of the timed launches
};

struct Span {
  std::string name;
  hipEvent_t a, b;
  double flops, bytes;
};

}  // namespace

namespace {
// Device storage shared by the prefixes made in one call: their KV store and
// their final hidden states; freed with the last of those prefixes.
struct KvStore {
  uint16_t* kv = nullptr;     // per layer K [cap][nkv][hd], V^T [nkv][hd][cap]
  float* hidden = nullptr;    // [n][d]
  int refs = 0;
};
}  // namespace

struct lmop_prefix {
  lmop_ctx* ctx = nullptr;
  lmop_prefix* parent = nullptr;
  int n = 0;       // own tokens
  int start = 0;   // tokens of the parent chain
  int cap = 0;     // slots of the KV store (a multiple of 64)
  int slot0 = 0;   // slot of the prefix's first token in the store (a multiple of 8)
  KvStore* store = nullptr;
  uint16_t* kv = nullptr;     // = store->kv
  float* hidden = nullptr;    // device [d]: last token's final-layer hidden state
  int children = 0;
  bool released = false;
  uint64_t generation = 0;
  int64_t id = 0;
};

struct lmop_ctx {
  lmop_config cfg{};
  int device = -1;
  bool host_only = false;
  hipStream_t stream = nullptr;
  bool own_stream = false;
  std::string err;
  bool dead = false;
  // testing hook (LMOP_INJECT_LAUNCH_FAILURE=<name>:<n>): the n-th launch
  // timed under <name> fails as a HIP launch error would, without launching
  std::string inject_name;
  long inject_at = 0, inject_count = 0;
  // set by lmop_plan_rows: eval_rows_impl stops after planning and fills it
  lmop_eval_plan* plan_out = nullptr;
  bool loaded = false;
  uint64_t generation = 0;
  int64_t next_prefix_id = 1;

  // dims
  int nq_dim = 0, nkv_dim = 0, qkv_n = 0, f64 = 0;
  uint32_t wfmt = LMOP_W_INT4_G32;  // format of the loaded linear maps

  // weights (device)
  uint16_t* emb = nullptr;
  uint16_t* head = nullptr;
  float* final_norm = nullptr;
  std::vector<LayerW> layers;
  std::vector<void*> weight_allocs;
  float2* rope_tab = nullptr;

  // library-allocated scratch: named grow-only buffers
  std::map<std::string, std::pair<void*, size_t>> ws;

  // device memory the library allocated itself (weights, prefix KV stores,
  // scratch), with its peak since lmop_create
  std::unordered_map<void*, size_t> alloc_sz;
  size_t dev_bytes = 0, dev_peak = 0;
  // the caller's workspace (lmop_set_workspace) and the most of it one call used
  char* user_ws = nullptr;
  size_t user_ws_bytes = 0, user_ws_peak = 0;
  // While a call runs with `carving` set, every scratch buffer is a fixed
  // region of [carve_base, carve_base + carve_size) laid out up front for the
  // call (`carved`); carve_base is the caller's workspace or the library's
  // static no-allocation array (a host-only ctx plans against the size
  // alone).
  bool carving = false;
  char* carve_base = nullptr;
  size_t carve_size = 0;
  std::map<std::string, std::pair<void*, size_t>> carved;
  // the current call allocates nothing: no device memory, no pinned host
  // memory, no events
  bool no_alloc = false;
  // device address of the static no-allocation array on this ctx's device
  void* static_scratch = nullptr;

  std::set<lmop_prefix*> prefixes;

  // pinned host staging for batch uploads and result readback: two slots, so
  // that one batch's host-side packing overlaps the previous batch on the GPU.
  // A no-allocation call stages through ordinary host memory instead.
  struct Staging {
    char* p = nullptr;          // pinned buffer
    size_t bytes = 0;
    std::vector<char> host;     // pageable buffer of no-allocation calls
    char* cur = nullptr;        // the buffer of the current use
    size_t cur_bytes = 0;
    size_t used = 0;            // bump offset within the current use
    hipEvent_t done = nullptr;  // recorded after the slot's last device access
    bool pending = false;
  };
  Staging stage[2];

  // profiling
  int32_t prof = 0;  // 0: off; N: every N-th launch of each kernel is timed
  std::vector<hipEvent_t> ev_free;
  std::vector<Span> spans;
  std::map<std::string, Stat> stats;
};

namespace {

lmop_status fail(lmop_ctx* c, lmop_status st, const char* fmt, ...) {
  if (c) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    c->err = buf;
    if (st == LMOP_ERR_DEVICE) c->dead = true;
  }
  return st;
}

#define HIP_OK(ctx, call)                                                                   \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return fail(ctx, e_ == hipErrorOutOfMemory ? LMOP_ERR_OOM : LMOP_ERR_DEVICE,          \
                  "%s failed: %s (%s:%d)", #call, hipGetErrorString(e_), __FILE__, __LINE__); \
  } while (0)

#define LMOP_TRY(expr)                \
  do {                                \
    lmop_status s_ = (expr);          \
    if (s_ != LMOP_OK) return s_;     \
  } while (0)

lmop_status dev_alloc(lmop_ctx* c, void** p, size_t bytes) {
  *p = nullptr;
  if (c->no_alloc)
    return fail(c, LMOP_ERR_STATE, "internal: a no-allocation call asked for %zu bytes", bytes);
  if (bytes == 0) bytes = 256;
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return fail(c, LMOP_ERR_OOM, "hipMalloc(%zu bytes) failed: %s", bytes, hipGetErrorString(e));
  }
  c->alloc_sz[*p] = bytes;
  c->dev_bytes += bytes;
  c->dev_peak = std::max(c->dev_peak, c->dev_bytes);
  return LMOP_OK;
}

// frees an allocation of dev_alloc (NULL is a no-op)
hipError_t dev_free(lmop_ctx* c, void* p) {
  if (!p) return hipSuccess;
  auto it = c->alloc_sz.find(p);
  if (it != c->alloc_sz.end()) {
    c->dev_bytes -= it->second;
    c->alloc_sz.erase(it);
  }
  return hipFree(p);
}

// scratch buffers start on 256-byte boundaries and are at least 256 bytes
size_t scratch_round(size_t bytes) { return std::max<size_t>((bytes + 255) & ~(size_t)255, 256); }

// Named scratch buffer of at least `count` elements.  Library-allocated
// scratch grows and is kept (`zero` clears it whenever it is allocated);
// carved scratch is the region the call's plan reserved under that name.
template <typename T>
lmop_status ws_get(lmop_ctx* c, const char* name, size_t count, T** out, bool zero = false) {
  const size_t bytes = scratch_round(count * sizeof(T));
  if (c->carving) {
    auto it = c->carved.find(name);
    if (it == c->carved.end() || it->second.second < bytes)
      return fail(c, LMOP_ERR_STATE, "internal: the scratch plan has no %zu bytes for '%s'",
                  bytes, name);
    *out = (T*)it->second.first;
    return LMOP_OK;
  }
  auto& slot = c->ws[name];
  if (slot.second < bytes) {
    if (slot.first) {
      HIP_OK(c, hipStreamSynchronize(c->stream));
      HIP_OK(c, dev_free(c, slot.first));
    }
    slot = {nullptr, 0};
    size_t want = scratch_round(bytes + bytes / 4);
    void* p = nullptr;
    LMOP_TRY(dev_alloc(c, &p, want));
    slot = {p, want};
    if (zero) HIP_OK(c, launch_fill_u32(c->stream, p, want / 4, 0u));
  }
  *out = (T*)slot.first;
  return LMOP_OK;
}

// Releases one library-allocated scratch buffer (after the stream is idle).
lmop_status ws_release(lmop_ctx* c, const char* name) {
  auto it = c->ws.find(name);
  if (it == c->ws.end()) return LMOP_OK;
  HIP_OK(c, hipStreamSynchronize(c->stream));
  HIP_OK(c, dev_free(c, it->second.first));
  c->ws.erase(it);
  return LMOP_OK;
}

lmop_status ws_release_all(lmop_ctx* c) {
  if (c->ws.empty()) return LMOP_OK;
  HIP_OK(c, hipStreamSynchronize(c->stream));
  for (auto& kv : c->ws) HIP_OK(c, dev_free(c, kv.second.first));
  c->ws.clear();
  return LMOP_OK;
}

// ---------------------------------------------------------------- staging
// Makes slot `k` ready for a new batch of at most `need` bytes: waits until
// the device is done with its previous contents, grows it if needed.
lmop_status stage_begin(lmop_ctx* c, int k, size_t need) {
  auto& st = c->stage[k];
  if (st.pending) {
    HIP_OK(c, hipEventSynchronize(st.done));
    st.pending = false;
  }
  if (!st.done) {
    if (c->no_alloc)
      return fail(c, LMOP_ERR_STATE, "internal: staging event missing in a no-allocation call");
    HIP_OK(c, hipEventCreateWithFlags(&st.done, hipEventDisableTiming));
  }
  if (c->no_alloc) {
    // ordinary host memory: the copies from and to it are ordered by the
    // slot's event like the pinned ones
    if (st.host.size() < need + 16) st.host.resize(need + need / 4 + 16);
    st.cur = (char*)(((uintptr_t)st.host.data() + 15) & ~(uintptr_t)15);
    st.cur_bytes = st.host.size() - (size_t)(st.cur - st.host.data());
  } else {
    if (st.bytes < need) {
      if (st.p) HIP_OK(c, hipHostFree(st.p));
      st.p = nullptr;
      st.bytes = 0;
      const size_t want = need + need / 4;
      void* q = nullptr;
      HIP_OK(c, hipHostMalloc(&q, want, hipHostMallocDefault));
      st.p = (char*)q;
      st.bytes = want;
    }
    st.cur = st.p;
    st.cur_bytes = st.bytes;
  }
  st.used = 0;
  return LMOP_OK;
}

// Copies n elements into slot k (16-byte aligned) and returns the staged copy.
template <typename T>
lmop_status stage_put(lmop_ctx* c, int k, const T* src, size_t n, T** out) {
  auto& st = c->stage[k];
  const size_t off = (st.used + 15) & ~(size_t)15;
  if (off + n * sizeof(T) > st.cur_bytes)
    return fail(c, LMOP_ERR_STATE, "internal: staging slot overflow (%zu + %zu > %zu)", off,
                n * sizeof(T), st.cur_bytes);
  *out = (T*)(st.cur + off);
  if (src && n) std::memcpy(*out, src, n * sizeof(T));
  st.used = off + n * sizeof(T);
  return LMOP_OK;
}

// The device has been handed everything that reads or writes slot k.
lmop_status stage_mark(lmop_ctx* c, int k) {
  auto& st = c->stage[k];
  HIP_OK(c, hipEventRecord(st.done, c->stream));
  st.pending = true;
  return LMOP_OK;
}

// Upper bound of the staging bytes one batch of T tokens and R rows needs.
size_t stage_need(int T, int R, size_t n_work) {
  // tokens, positions, slots; per row: attention row, last-token index,
  // head row pointer, automaton state, pick; work items; alignment
  return (size_t)T * 12 + (size_t)R * (sizeof(AttnRow) + 8 + sizeof(void*) + sizeof(HeadPick)) +
         n_work * sizeof(int2) + 16 * 17;
}

// ---------------------------------------------------------------- profiling
// Timing events are only read for elapsed times, so they are recorded
// without the system-scope fence (a cache writeback and invalidate at every
// record, which with two events per kernel both slowed the step and
// perturbed the timed kernels).
hipEvent_t take_event(lmop_ctx* c) {
  if (!c->ev_free.empty()) {
    hipEvent_t e = c->ev_free.back();
    c->ev_free.pop_back();
    return e;
  }
  if (c->no_alloc) return nullptr;  // that launch is counted, not timed
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

template <typename F>
lmop_status timed(lmop_ctx* c, const char* name, double flops, double bytes, F&& launch) {
  hipEvent_t a = nullptr, b = nullptr;
  if (c->prof > 0 && c->stats[name].launches++ % c->prof == 0) {
    a = take_event(c);
    b = take_event(c);
    if (a && b) {
      HIP_OK(c, hipEventRecord(a, c->stream));
    } else {
      if (a) c->ev_free.push_back(a);
      if (b) c->ev_free.push_back(b);
      a = b = nullptr;
    }
  }
  if (!c->inject_name.empty() && c->inject_name == name && ++c->inject_count == c->inject_at)
    return fail(c, LMOP_ERR_DEVICE, "launch of %s failed: injected failure", name);
  hipError_t e = launch();
  if (e != hipSuccess) return fail(c, LMOP_ERR_DEVICE, "launch of %s failed: %s", name,
                                   hipGetErrorString(e));
  if (a && b) {
    HIP_OK(c, hipEventRecord(b, c->stream));
    c->spans.push_back(Span{name, a, b, flops, bytes});
  }
  return LMOP_OK;
}

lmop_status resolve_spans(lmop_ctx* c) {
  for (auto& s : c->spans) {
    HIP_OK(c, hipEventSynchronize(s.b));
    float ms = 0.f;
    HIP_OK(c, hipEventElapsedTime(&ms, s.a, s.b));
    Stat& st = c->stats[s.name];
    st.timed += 1;
    st.ms += ms;
    st.flops += s.flops;
    st.bytes += s.bytes;
    c->ev_free.push_back(s.a);
    c->ev_free.push_back(s.b);
  }
  c->spans.clear();
  return LMOP_OK;
}

lmop_status sync(lmop_ctx* c) {
  HIP_OK(c, hipStreamSynchronize(c->stream));
  return resolve_spans(c);
}

// ---------------------------------------------------------------- validation
lmop_status check_config(const lmop_config* cfg, lmop_ctx* c) {
  if (!cfg) return fail(c, LMOP_ERR_INVALID_ARG, "config is NULL");
  if (cfg->n_layers < 0 || cfg->d_model <= 0 || cfg->n_heads <= 0 || cfg->n_kv_heads <= 0 ||
      cfg->head_dim <= 0 || cfg->d_ff <= 0 || cfg->vocab <= 1 || !(cfg->rms_eps >= 0.f) ||
      !(cfg->rope_theta > 0.f) || cfg->max_seq < 0)
    return fail(c, LMOP_ERR_INVALID_ARG, "config has a non-positive dimension or parameter");
  if (cfg->max_seq > kMaxSeq)
    return fail(c, LMOP_ERR_UNSUPPORTED, "max_seq %d (at most %d)", cfg->max_seq, kMaxSeq);
  if (cfg->head_dim != 64 && cfg->head_dim != 128)
    return fail(c, LMOP_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", cfg->head_dim);
  if (cfg->n_heads % cfg->n_kv_heads != 0)
    return fail(c, LMOP_ERR_UNSUPPORTED, "n_heads %% n_kv_heads != 0");
  if (cfg->d_model % 64 != 0)
    return fail(c, LMOP_ERR_UNSUPPORTED, "d_model %d is not a multiple of 64", cfg->d_model);
  if (cfg->group_size != 32)
    return fail(c, LMOP_ERR_UNSUPPORTED, "group_size %d (supported: 32)", cfg->group_size);
  if (cfg->vocab >= (1 << 24)) return fail(c, LMOP_ERR_UNSUPPORTED, "vocab too large");
  return LMOP_OK;
}

lmop_status check_qmat(lmop_ctx* c, const char* what, int layer, const lmop_qmat& m, int n,
                       int k) {
  if (!m.qweight || !m.scales)
    return fail(c, LMOP_ERR_INVALID_ARG, "layer %d %s: NULL qweight/scales", layer, what);
  if (m.n != n || m.k != k)
    return fail(c, LMOP_ERR_INVALID_ARG, "layer %d %s: shape [%d][%d], expected [%d][%d]", layer,
                what, m.n, m.k, n, k);
  return LMOP_OK;
}

bool prefix_live(const lmop_ctx* c, const lmop_prefix* p) {
  return p && c->prefixes.count(const_cast<lmop_prefix*>(p)) && !p->released &&
         p->generation == c->generation;
}

int prefix_total(const lmop_prefix* p) { return p ? p->start + p->n : 0; }

lmop_status check_tokens(lmop_ctx* c, const int32_t* t, int64_t n, const char* what) {
  const int V = c->cfg.vocab;
  for (int64_t i = 0; i < n; ++i)
    if (t[i] < 0 || t[i] >= V)
      return fail(c, LMOP_ERR_INVALID_ARG, "%s token %lld = %d outside [0, %d)", what,
                  (long long)i, t[i], V);
  return LMOP_OK;
}

// A token automaton's validity (the limits stated with lmop_automaton).
lmop_status check_automaton(lmop_ctx* c, const lmop_type* ty) {
  const lmop_automaton* a = ty->automaton;
  if (!a) return fail(c, LMOP_ERR_INVALID_ARG, "AUTOMATON type without an automaton");
  if (ty->max_tokens < 1 || ty->max_tokens > 8)
    return fail(c, LMOP_ERR_INVALID_ARG, "AUTOMATON max_tokens %d outside 1..8", ty->max_tokens);
  const int S = a->n_states;
  if (S < 1 || S > 65536)
    return fail(c, LMOP_ERR_INVALID_ARG, "automaton n_states %d outside 1..65536", S);
  if (!a->edge_offset || !a->edge_token || !a->edge_next || !a->accepting)
    return fail(c, LMOP_ERR_INVALID_ARG, "automaton has a NULL array");
  if (a->edge_offset[0] != 0) return fail(c, LMOP_ERR_INVALID_ARG, "automaton edge_offset[0] != 0");
  for (int s = 0; s < S; ++s)
    if (a->edge_offset[s + 1] < a->edge_offset[s])
      return fail(c, LMOP_ERR_INVALID_ARG, "automaton edge_offset decreases at state %d", s);
  const int E = a->edge_offset[S];
  if (E < 1 || E > (1 << 20))
    return fail(c, LMOP_ERR_INVALID_ARG, "automaton has %d edges (1..2^20)", E);
  LMOP_TRY(check_tokens(c, a->edge_token, E, "automaton edge"));
  std::set<int32_t> all;
  for (int s = 0; s < S; ++s) {
    const int e0 = a->edge_offset[s], e1 = a->edge_offset[s + 1];
    if (e0 == e1 && (s == 0 || !a->accepting[s]))
      return fail(c, LMOP_ERR_INVALID_ARG, "automaton state %d has no edges and %s", s,
                  s == 0 ? "is the start" : "is not accepting");
    std::set<int32_t> own;
    for (int e = e0; e < e1; ++e) {
      if (a->edge_next[e] < 0 || a->edge_next[e] >= S)
        return fail(c, LMOP_ERR_INVALID_ARG, "automaton edge %d leads to state %d", e,
                    a->edge_next[e]);
      if (!own.insert(a->edge_token[e]).second)
        return fail(c, LMOP_ERR_INVALID_ARG, "automaton state %d repeats token %d", s,
                    a->edge_token[e]);
      all.insert(a->edge_token[e]);
    }
  }
  if (ty->eos_token >= 0) {
    if (ty->eos_token >= c->cfg.vocab)
      return fail(c, LMOP_ERR_INVALID_ARG, "eos_token %d outside the vocabulary", ty->eos_token);
    if (all.count(ty->eos_token))
      return fail(c, LMOP_ERR_INVALID_ARG, "eos_token %d is an edge token", ty->eos_token);
  }
  const size_t n_union = all.size() + (ty->eos_token >= 0 ? 1 : 0);
  if (n_union > 4096)
    return fail(c, LMOP_ERR_INVALID_ARG, "automaton uses more than 4096 distinct tokens");
  if ((size_t)S * n_union > (size_t(1) << 26))
    return fail(c, LMOP_ERR_INVALID_ARG, "automaton states x distinct tokens exceeds 2^26");
  return LMOP_OK;
}

lmop_status check_type(lmop_ctx* c, const lmop_type* ty) {
  if (!ty) return fail(c, LMOP_ERR_INVALID_ARG, "type is NULL");
  if (ty->kind < LMOP_BOOL || ty->kind > LMOP_AUTOMATON)
    return fail(c, LMOP_ERR_INVALID_ARG, "unknown type kind %d", ty->kind);
  if (ty->kind == LMOP_AUTOMATON) return check_automaton(c, ty);
  if (!ty->tokens) return fail(c, LMOP_ERR_INVALID_ARG, "type tokens is NULL");
  const int n = ty->n_tokens;
  if (ty->kind == LMOP_BOOL && n != 2)
    return fail(c, LMOP_ERR_INVALID_ARG, "BOOL needs 2 tokens, got %d", n);
  if (ty->kind == LMOP_ENUM && (n < 1 || n > 4096))
    return fail(c, LMOP_ERR_INVALID_ARG, "ENUM needs 1..4096 tokens, got %d", n);
  if (ty->kind == LMOP_INT) {
    if (n != 10) return fail(c, LMOP_ERR_INVALID_ARG, "INT needs 10 digit tokens, got %d", n);
    if (ty->max_tokens < 1 || ty->max_tokens > 8)
      return fail(c, LMOP_ERR_INVALID_ARG, "INT max_tokens %d outside 1..8", ty->max_tokens);
    if (ty->eos_token < 0 || ty->eos_token >= c->cfg.vocab)
      return fail(c, LMOP_ERR_INVALID_ARG, "INT eos_token %d outside the vocabulary",
                  ty->eos_token);
  }
  LMOP_TRY(check_tokens(c, ty->tokens, n, "type"));
  std::set<int32_t> seen(ty->tokens, ty->tokens + n);
  if ((int)seen.size() != n) return fail(c, LMOP_ERR_INVALID_ARG, "type tokens are not distinct");
  if (ty->kind == LMOP_INT && seen.count(ty->eos_token))
    return fail(c, LMOP_ERR_INVALID_ARG, "INT eos_token is one of the digit tokens");
  return LMOP_OK;
}

// ---------------------------------------------------------------- dedup
uint64_t mix(uint64_t h, uint64_t v) {
  h ^= v + 0x9e3779b97f4a7c15ull + (h << 6) + (h >> 2);
  return h * 0xff51afd7ed558ccdull;
}

void dedup(const int32_t* tokens, const int64_t* offsets, int n_rows, const int64_t* keys,
           int32_t* rep, int32_t* n_unique) {
  std::unordered_map<uint64_t, std::vector<int32_t>> buckets;
  buckets.reserve((size_t)n_rows * 2);
  int u = 0;
  for (int r = 0; r < n_rows; ++r) {
    const int64_t b = offsets[r], e = offsets[r + 1];
    uint64_t h = mix(0x1234567ull, (uint64_t)(keys ? keys[r] : 0));
    h = mix(h, (uint64_t)(e - b));
    for (int64_t i = b; i < e; ++i) h = mix(h, (uint32_t)tokens[i]);
    auto& cand = buckets[h];
    int found = -1;
    for (int32_t q : cand) {
      const int64_t qb = offsets[q], qe = offsets[q + 1];
      if ((keys ? keys[q] : 0) != (keys ? keys[r] : 0)) continue;
      if (qe - qb != e - b) continue;
      if (std::equal(tokens + b, tokens + e, tokens + qb)) {
        found = q;
        break;
      }
    }
    if (found < 0) {
      cand.push_back(r);
      rep[r] = r;
      ++u;
    } else {
      rep[r] = found;
    }
  }
  *n_unique = u;
}

// ---------------------------------------------------------------- weights
lmop_status upload(lmop_ctx* c, const void* src, size_t bytes, bool on_device, void** dst) {
  LMOP_TRY(dev_alloc(c, dst, bytes));
  c->weight_allocs.push_back(*dst);
  HIP_OK(c, hipMemcpyAsync(*dst, src, bytes,
                           on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice,
                           c->stream));
  return LMOP_OK;
}

void free_weights(lmop_ctx* c) {
  for (void* p : c->weight_allocs) (void)dev_free(c, p);
  c->weight_allocs.clear();
  c->layers.clear();
  c->emb = c->head = nullptr;
  c->final_norm = nullptr;
}

// Packs up to three source matrices (rows = output columns) into one tiled
// int4 weight.  colmap[j] = (source << 24) | row, or -1 for a zero column.
lmop_status pack_fp8(lmop_ctx* c, const lmop_qmat* const* srcs, int n_src,
                     const std::vector<int32_t>& colmap, int n_logical, int k, bool on_device,
                     PackedW* out);

lmop_status pack(lmop_ctx* c, const lmop_qmat* const* srcs, int n_src, const std::vector<int32_t>& colmap,
                 int n_logical, int k, bool on_device, PackedW* out) {
  if (c->wfmt == LMOP_W_FP8_E4M3)
    return pack_fp8(c, srcs, n_src, colmap, n_logical, k, on_device, out);
  PackedW w;
  w.n = n_logical;
  w.np = (int)colmap.size();
  w.k = k;
  w.kp = round_up(k, 64);
  const int kg = w.kp / 32;
  void* qp = nullptr;
  void* sp = nullptr;
  LMOP_TRY(dev_alloc(c, &qp, (size_t)(w.np / 64) * kg * 1024));
  c->weight_allocs.push_back(qp);
  LMOP_TRY(dev_alloc(c, &sp, (size_t)(w.np / 64) * kg * 128));
  c->weight_allocs.push_back(sp);
  w.qpack = (uint32_t*)qp;
  w.spack = (half_bits*)sp;

  RepackSrc rs{};
  std::vector<void*> staging;
  for (int i = 0; i < n_src; ++i) {
    const lmop_qmat& m = *srcs[i];
    const int kps = round_up(m.k, 32);
    rs.kp_src[i] = kps;
    if (on_device) {
      rs.q[i] = m.qweight;
      rs.s[i] = (const half_bits*)m.scales;
    } else {
      void* dq = nullptr;
      void* ds = nullptr;
      LMOP_TRY(dev_alloc(c, &dq, (size_t)m.n * kps / 2));
      staging.push_back(dq);
      LMOP_TRY(dev_alloc(c, &ds, (size_t)m.n * (kps / 32) * 2));
      staging.push_back(ds);
      HIP_OK(c, hipMemcpyAsync(dq, m.qweight, (size_t)m.n * kps / 2, hipMemcpyHostToDevice,
                               c->stream));
      HIP_OK(c, hipMemcpyAsync(ds, m.scales, (size_t)m.n * (kps / 32) * 2,
                               hipMemcpyHostToDevice, c->stream));
      rs.q[i] = (const uint8_t*)dq;
      rs.s[i] = (const half_bits*)ds;
    }
  }
  void* dmap = nullptr;
  LMOP_TRY(dev_alloc(c, &dmap, colmap.size() * 4));
  staging.push_back(dmap);
  HIP_OK(c, hipMemcpyAsync(dmap, colmap.data(), colmap.size() * 4, hipMemcpyHostToDevice,
                           c->stream));
  LMOP_TRY(timed(c, "repack_w4", 0, 0, [&] { return launch_repack_w4(c->stream, rs, (const int32_t*)dmap, w); }));
  HIP_OK(c, hipStreamSynchronize(c->stream));
  for (void* p : staging) HIP_OK(c, dev_free(c, p));
  *out = w;
  return LMOP_OK;
}

// The same for FP8 weights: E4M3 codes [n][k] and fp32 row scales [n] of up
// to three sources -> 2 KB tiles per 64 columns x 32 features, fp32 scales in
// packed column order.
lmop_status pack_fp8(lmop_ctx* c, const lmop_qmat* const* srcs, int n_src,
                     const std::vector<int32_t>& colmap, int n_logical, int k, bool on_device,
                     PackedW* out) {
  PackedW w;
  w.n = n_logical;
  w.np = (int)colmap.size();
  w.k = k;
  w.kp = round_up(k, 64);
  const int kg = w.kp / 32;
  void* qp = nullptr;
  void* sp = nullptr;
  LMOP_TRY(dev_alloc(c, &qp, (size_t)(w.np / 64) * kg * 2048));
  c->weight_allocs.push_back(qp);
  LMOP_TRY(dev_alloc(c, &sp, (size_t)w.np * 4));
  c->weight_allocs.push_back(sp);
  w.qpack = (uint32_t*)qp;
  w.sscale = (float*)sp;
  RepackSrc rs{};
  std::vector<void*> staging;
  for (int i = 0; i < n_src; ++i) {
    const lmop_qmat& m = *srcs[i];
    rs.kp_src[i] = m.k;
    if (on_device) {
      rs.q[i] = m.qweight;
      rs.sf[i] = (const float*)m.scales;
    } else {
      void* dq = nullptr;
      void* ds = nullptr;
      LMOP_TRY(dev_alloc(c, &dq, (size_t)m.n * m.k));
      staging.push_back(dq);
      LMOP_TRY(dev_alloc(c, &ds, (size_t)m.n * 4));
      staging.push_back(ds);
      HIP_OK(c, hipMemcpyAsync(dq, m.qweight, (size_t)m.n * m.k, hipMemcpyHostToDevice,
                               c->stream));
      HIP_OK(c, hipMemcpyAsync(ds, m.scales, (size_t)m.n * 4, hipMemcpyHostToDevice, c->stream));
      rs.q[i] = (const uint8_t*)dq;
      rs.sf[i] = (const float*)ds;
    }
  }
  void* dmap = nullptr;
  LMOP_TRY(dev_alloc(c, &dmap, colmap.size() * 4));
  staging.push_back(dmap);
  HIP_OK(c, hipMemcpyAsync(dmap, colmap.data(), colmap.size() * 4, hipMemcpyHostToDevice,
                           c->stream));
  LMOP_TRY(timed(c, "repack_w8", 0, 0,
                 [&] { return launch_repack_w8(c->stream, rs, (const int32_t*)dmap, w); }));
  HIP_OK(c, hipStreamSynchronize(c->stream));
  for (void* p : staging) HIP_OK(c, dev_free(c, p));
  *out = w;
  return LMOP_OK;
}

// The GEMM of a packed linear map in the loaded weight format.
hipError_t launch_gemm_packed(const lmop_ctx* c, GemmArgs& ga, const PackedW& W, int epi) {
  ga.bq = W.qpack;
  if (c->wfmt == LMOP_W_FP8_E4M3) {
    ga.bsc = W.sscale;
    return launch_gemm_w8(c->stream, ga, epi);
  }
  ga.bs = W.spack;
  return launch_gemm_w4(c->stream, ga, epi);
}

// timing names and weight bytes per parameter of the loaded format
const char* gemm_name(const lmop_ctx* c, const char* proj, bool decode = false) {
  static thread_local std::string n;
  n = std::string(decode ? "decode_" : "") +
      (c->wfmt == LMOP_W_FP8_E4M3 ? "gemm_w8a16_" : "gemm_w4a16_") + proj;
  return n.c_str();
}
double weight_bytes(const lmop_ctx* c, double n, double k) {
  return c->wfmt == LMOP_W_FP8_E4M3 ? n * k + n * 4 : n * k * 0.5625;
}

std::vector<int32_t> concat_map(const int* rows, int n_parts, int np) {
  std::vector<int32_t> m(np, -1);
  int j = 0;
  for (int s = 0; s < n_parts; ++s)
    for (int r = 0; r < rows[s]; ++r) m[j++] = (s << 24) | r;
  return m;
}

// ---------------------------------------------------------------- scratch plan
// own-KV slots: each row starts at a multiple of 8 (16-byte aligned V^T runs);
// the store has 64 spare slots so a row's last 64-key block stays in bounds
int own_store_cap(int used) { return round_up(used + 64, 64); }

// The largest sizes one call's scratch buffers reach.  A call computes its
// plan before any device work, so that scratch carved from a caller's
// workspace (or the static no-allocation array) is laid out once, and
// library-allocated scratch is grown once.
struct Need {
  size_t T = 0, R = 0, W = 0;  // tokens, rows, attention work items of one forward pass
  size_t last = 0;             // tokens whose final hidden state one pass keeps
  size_t own_kv = 0;           // bytes of the own-KV store
  size_t head_rows = 0;        // rows of one head pass (0: no head)
  bool restricted = false;     // restricted head: no vocabulary partials
  bool dump = false;           // a [head_rows][vocab] logit dump
  size_t n_sel = 0;            // allowed-token list (0: no type tables)
  size_t state_mask = 0;       // bytes of the automaton's state-mask table
};

// (name, bytes) of every scratch buffer of a call with these maxima, in
// layout order; the names are the ones ws_get asks for
std::vector<std::pair<const char*, size_t>> scratch_items(const lmop_ctx* c, const Need& n) {
  const size_t d = c->cfg.d_model, V = c->cfg.vocab;
  const size_t n_chunks = (V + kHeadVocabChunk - 1) / kHeadVocabChunk;
  std::vector<std::pair<const char*, size_t>> it;
  auto add = [&](const char* name, size_t bytes) { it.emplace_back(name, scratch_round(bytes)); };
  // a batch whose rows all have empty suffixes still reads one row of x
  const size_t T = std::max<size_t>(n.T, 1);
  add("tok", T * 4);
  add("pos", T * 4);
  add("slot", T * 4);
  add("rows", n.R * sizeof(AttnRow));
  add("work", n.W * sizeof(int2));
  add("x", T * d * 4);
  add("h", T * d * 2);
  add("q", T * c->nq_dim * 2);
  add("att", T * c->nq_dim * 2);
  add("act", T * c->f64 * 2);
  add("last", n.last * 4);
  add("xlast", n.last * d * 4);
  add("attlast", n.last * c->nq_dim * 2);
  add("own_kv", n.own_kv);
  if (n.head_rows > 0) {
    const size_t R = n.head_rows;
    add("head_rowptr", R * sizeof(void*));
    add("head_hn", R * d * 2);
    add("head_part", n.restricted ? sizeof(float2) : R * n_chunks * sizeof(float2));
    add("head_zsel", R * n.n_sel * 4);
    add("head_pick", R * sizeof(HeadPick));
    add("head_state", R * 4);
    if (n.dump) add("dump", R * V * 4);
  }
  if (n.n_sel > 0) {
    add("sel", V * 4);
    add("allowed", n.n_sel * 4);
    if (n.state_mask > 0) add("state_mask", n.state_mask);
  }
  return it;
}

size_t scratch_total(const lmop_ctx* c, const Need& n) {
  size_t t = 0;
  for (auto& i : scratch_items(c, n)) t += i.second;
  return t;
}

// Lays out every scratch buffer of the call in the carved region, or grows
// the library-allocated ones to their largest size up front.  The own-KV
// store must hold finite values wherever attention reads past a row's keys
// (masked keys still multiply their values by 0), so carved memory, which
// may hold anything, is cleared.
lmop_status reserve_scratch(lmop_ctx* c, const Need& n) {
  const auto items = scratch_items(c, n);
  if (!c->carving) {
    for (auto& i : items) {
      char* p;
      LMOP_TRY(ws_get(c, i.first, i.second, &p, std::strcmp(i.first, "own_kv") == 0));
    }
    return LMOP_OK;
  }
  c->carved.clear();
  size_t off = 0;
  for (auto& i : items) {
    c->carved[i.first] = {c->carve_base + off, i.second};
    off += i.second;
  }
  if (off > c->carve_size)
    return fail(c, LMOP_ERR_OOM, "the call needs %zu bytes of scratch, the %s holds %zu", off,
                c->no_alloc ? "no-allocation array" : "workspace", c->carve_size);
  if (!c->no_alloc) c->user_ws_peak = std::max(c->user_ws_peak, off);
  auto kv = c->carved.find("own_kv");
  if (kv != c->carved.end())
    HIP_OK(c, launch_fill_u32(c->stream, kv->second.first, kv->second.second / 4, 0u));
  return LMOP_OK;
}

// Batches of consecutive entries within `budget` tokens and kMaxBatchRows
// entries; an entry longer than the budget forms a batch of its own.
std::vector<std::pair<size_t, size_t>> make_batches(const std::vector<int>& len, int budget) {
  std::vector<std::pair<size_t, size_t>> out;
  for (size_t u0 = 0; u0 < len.size();) {
    size_t u1 = u0;
    int T = 0;
    while (u1 < len.size() && (int)(u1 - u0) < kMaxBatchRows) {
      if (u1 > u0 && T + len[u1] > budget) break;
      T += len[u1];
      ++u1;
    }
    out.emplace_back(u0, u1);
    u0 = u1;
  }
  return out;
}

int attn_tiles(int n_q, int G) { return (n_q * G + ATTN_QTILE - 1) / ATTN_QTILE; }

// The forward-pass maxima of a list of batches over entries of len[]
void batch_need(const std::vector<int>& len, const std::vector<std::pair<size_t, size_t>>& batches,
                int G, Need* n) {
  for (auto& b : batches) {
    size_t T = 0, W = 0, last = 0;
    for (size_t u = b.first; u < b.second; ++u) {
      T += len[u];
      W += attn_tiles(len[u], G);
      last += len[u] > 0;
    }
    n->T = std::max(n->T, T);
    n->R = std::max(n->R, b.second - b.first);
    n->W = std::max(n->W, W);
    n->last = std::max(n->last, last);
  }
}

// Row batches and own-KV placement of one lmop_eval_rows call.
struct Schedule {
  std::vector<std::pair<size_t, size_t>> batches;  // ranges of the distinct rows
  std::vector<int> base_of, group_of;              // per batch: first slot, decode group
  std::vector<int> group_cap;                      // per group: slots of its store
  Need need;
  int budget = 0;
};

// Own-KV placement.  Integer and automaton types decode further tokens for
// a group of consecutive batches at once: the group's batches keep their KV
// in one store, so each decode step is one forward over all live rows of the
// group instead of one small forward per batch.  A group is bounded by
// `group_bytes`, by the store's slot limit and by the token budget (a decode
// step has one token per live row).  Single-step types need no KV after the
// first step: one batch per group.  Each row's slots start at a multiple of
// 8 and leave room for `dec` decoded tokens.
void make_groups(const std::vector<int>& len, int dec, int budget, size_t slot_bytes,
                 size_t group_bytes, Schedule* s) {
  const auto& batches = s->batches;
  const int n_batches = (int)batches.size();
  s->base_of.assign(n_batches, 0);
  s->group_of.assign(n_batches, 0);
  s->group_cap.clear();
  for (int b = 0; b < n_batches;) {
    int b1 = b, used = 0;
    size_t rows = 0;
    while (b1 < n_batches) {
      int slots = 0;
      for (size_t u = batches[b1].first; u < batches[b1].second; ++u)
        slots = round_up(slots + len[u] + dec, 8);
      const size_t r = batches[b1].second - batches[b1].first;
      if (b1 > b && (dec == 0 || (size_t)own_store_cap(used + slots) * slot_bytes > group_bytes ||
                     own_store_cap(used + slots) > kMaxStoreSlots || rows + r > (size_t)budget))
        break;
      s->base_of[b1] = used;
      s->group_of[b1] = (int)s->group_cap.size();
      used += slots;
      rows += r;
      ++b1;
    }
    s->group_cap.push_back(own_store_cap(used));
    b = b1;
  }
}

// Largest budget in [1, want] for which fits(budget) holds, trying `want`
// first; fits() keeps the plan of the budget it was last called with, so the
// winner is evaluated last.  0 if not even a budget of 1 fits.
template <typename F>
int fit_budget(int want, F&& fits) {
  if (fits(want)) return want;
  if (want <= 1 || !fits(1)) return 0;
  int lo = 1, hi = want;  // fits(lo), !fits(hi)
  while (hi - lo > 1) {
    const int mid = lo + (hi - lo) / 2;
    (fits(mid) ? lo : hi) = mid;
  }
  fits(lo);
  return lo;
}

// ---------------------------------------------------------------- forward
struct Batch {
  int T = 0;        // query tokens of this launch
  int R = 0;        // rows
  int n_work = 0;   // attention work items
  uint16_t* own_kv = nullptr;
  int own_cap = 0;
  // Tokens whose final hidden state is needed (ws "last"), or 0 = all tokens.
  // With n_last > 0 the last layer's O-projection and MLP run on those tokens
  // only, and their final hidden states land in ws "xlast" [n_last][d].
  int n_last = 0;
  // keys visible to the batch's query tokens, summed (for the attention FLOP count)
  double visible_keys = 0;
  // a decode step (one token per live row): its launches are timed under
  // "decode_"-prefixed names, apart from the prefill passes
  bool decode = false;
};

// One pass of all layers over the T tokens whose ids/positions/slots and row
// descriptors are already on the device (ws "tok", "pos", "slot", "rows", "work").
lmop_status forward(lmop_ctx* c, const Batch& b) {
  const lmop_config& cf = c->cfg;
  const int T = b.T, d = cf.d_model, hd = cf.head_dim;
  if (T == 0) return LMOP_OK;
  int32_t *tok, *pos, *slot;
  AttnRow* rows;
  int2* work;
  float* x;
  uint16_t *h, *q, *att, *act;
  LMOP_TRY(ws_get(c, "tok", T, &tok));
  LMOP_TRY(ws_get(c, "pos", T, &pos));
  LMOP_TRY(ws_get(c, "slot", T, &slot));
  LMOP_TRY(ws_get(c, "rows", b.R, &rows));
  LMOP_TRY(ws_get(c, "work", b.n_work, &work));
  LMOP_TRY(ws_get(c, "x", (size_t)T * d, &x));
  LMOP_TRY(ws_get(c, "h", (size_t)T * d, &h));
  LMOP_TRY(ws_get(c, "q", (size_t)T * c->nq_dim, &q));
  LMOP_TRY(ws_get(c, "att", (size_t)T * c->nq_dim, &att));
  LMOP_TRY(ws_get(c, "act", (size_t)T * c->f64, &act));

  LMOP_TRY(timed(c, "embed", 0, (double)T * d * 6, [&] {
    return launch_embed(c->stream, tok, T, c->emb, d, x);
  }));
  const size_t kv_layer = (size_t)2 * b.own_cap * c->nkv_dim;
  for (int l = 0; l < cf.n_layers; ++l) {
    const LayerW& L = c->layers[l];
    const double nbytes_norm = (double)T * d * 6;
    LMOP_TRY(timed(c, b.decode ? "decode_rmsnorm" : "rmsnorm", 0, nbytes_norm, [&] {
      return launch_rmsnorm(c->stream, x, d, nullptr, T, L.attn_norm, d, cf.rms_eps, h, d);
    }));
    uint16_t* kc = b.own_kv + l * kv_layer;
    uint16_t* vt = kc + (size_t)b.own_cap * c->nkv_dim;
    {
      GemmArgs ga{};
      ga.A = h;
      ga.lda = d;
      ga.M = T;
      ga.N = L.qkv.np;
      ga.K = L.qkv.kp;
      ga.pos = pos;
      ga.slot = slot;
      ga.rope = c->rope_tab;
      ga.qout = q;
      ga.kc = kc;
      ga.vt = vt;
      ga.cap = b.own_cap;
      ga.nq = cf.n_heads;
      ga.nkv = cf.n_kv_heads;
      ga.hd = hd;
      const double flops = 2.0 * T * L.qkv.n * L.qkv.k;
      const double bytes = (double)T * L.qkv.k * 2 + weight_bytes(c, L.qkv.n, L.qkv.k) +
                           (double)T * L.qkv.n * 2;
      LMOP_TRY(timed(c, gemm_name(c, "qkv", b.decode), flops, bytes,
                     [&] { return launch_gemm_packed(c, ga, L.qkv, EPI_QKV); }));
    }
    AttnArgs aa{};
    aa.q = q;
    aa.ldq = c->nq_dim;
    aa.out = att;
    aa.ldo = c->nq_dim;
    aa.rows = rows;
    aa.work = work;
    aa.n_work = b.n_work;
    aa.own_kv = b.own_kv;
    aa.own_cap = b.own_cap;
    aa.layer = l;
    aa.nq = cf.n_heads;
    aa.nkv = cf.n_kv_heads;
    aa.hd = hd;
    // per visible (query token, key) pair and query head: q.k and p.v, 2 FLOP per dim each
    const double attn_flops = 4.0 * hd * cf.n_heads * b.visible_keys;
    LMOP_TRY(timed(c, b.decode ? "decode_attention" : "attention", attn_flops, 0,
                   [&] { return launch_attention(c->stream, aa); }));
    // in the last layer only the selected tokens continue (their K/V are written above)
    int M = T;
    float* xr = x;
    uint16_t* ar = att;
    if (l == cf.n_layers - 1 && b.n_last > 0) {
      int32_t* last;
      LMOP_TRY(ws_get(c, "last", b.n_last, &last));
      LMOP_TRY(ws_get(c, "xlast", (size_t)b.n_last * d, &xr));
      LMOP_TRY(ws_get(c, "attlast", (size_t)b.n_last * c->nq_dim, &ar));
      LMOP_TRY(timed(c, "gather_rows", 0, (double)b.n_last * (d * 8 + c->nq_dim * 4), [&] {
        return launch_gather_rows(c->stream, last, b.n_last, x, d, xr, att, c->nq_dim, ar);
      }));
      M = b.n_last;
    }
    auto gemm2 = [&](const char* name, const void* A, int lda, const PackedW& W, int epi,
                     void* C, int ldc, int n_out) {
      GemmArgs ga{};
      ga.A = A;
      ga.lda = lda;
      ga.M = M;
      ga.N = W.np;
      ga.K = W.kp;
      ga.C = C;
      ga.ldc = ldc;
      ga.n_out = n_out;
      ga.X = xr;
      ga.ldx = d;
      const double flops = 2.0 * M * W.n * W.k;
      const double bytes = (double)M * W.k * 2 + weight_bytes(c, W.n, W.k) +
                           (double)M * W.n * (epi == EPI_ADD_F32 ? 8 : 2);
      return timed(c, gemm_name(c, name, b.decode), flops, bytes,
                   [&] { return launch_gemm_packed(c, ga, W, epi); });
    };
    LMOP_TRY(gemm2("o", ar, c->nq_dim, L.o, EPI_ADD_F32, nullptr, 0, d));
    LMOP_TRY(timed(c, b.decode ? "decode_rmsnorm" : "rmsnorm", 0, (double)M * d * 6, [&] {
      return launch_rmsnorm(c->stream, xr, d, nullptr, M, L.mlp_norm, d, cf.rms_eps, h, d);
    }));
    LMOP_TRY(gemm2("gateup", h, d, L.gu, EPI_SWIGLU, act, c->f64, c->f64));
    LMOP_TRY(gemm2("down", act, c->f64, L.down, EPI_ADD_F32, nullptr, 0, d));
  }
  return LMOP_OK;
}

// Uploads host-built per-token and per-row arrays for one forward pass
// through staging slot k (which stage_begin has sized); does not wait.
lmop_status upload_batch(lmop_ctx* c, int k, const std::vector<int32_t>& tok,
                         const std::vector<int32_t>& pos, const std::vector<int32_t>& slot,
                         const std::vector<AttnRow>& rows, const std::vector<int2>& work,
                         const std::vector<int32_t>& last = {}) {
  c->stage[k].used = 0;
  auto put = [&](const char* name, const auto& v) -> lmop_status {
    using T = typename std::decay_t<decltype(v)>::value_type;
    T* d;
    T* h;
    LMOP_TRY(ws_get(c, name, v.size(), &d));
    if (v.empty()) return LMOP_OK;
    LMOP_TRY(stage_put(c, k, v.data(), v.size(), &h));
    HIP_OK(c, hipMemcpyAsync(d, h, v.size() * sizeof(T), hipMemcpyHostToDevice, c->stream));
    return LMOP_OK;
  };
  if (!last.empty()) LMOP_TRY(put("last", last));
  LMOP_TRY(put("tok", tok));
  LMOP_TRY(put("pos", pos));
  LMOP_TRY(put("slot", slot));
  LMOP_TRY(put("rows", rows));
  LMOP_TRY(put("work", work));
  return LMOP_OK;
}

void fill_segments(const lmop_prefix* p, AttnRow& r) {
  r.seg_kv[0] = r.seg_kv[1] = nullptr;
  r.seg_n[0] = r.seg_n[1] = 0;
  r.seg_cap[0] = r.seg_cap[1] = 0;
  r.seg_start[0] = r.seg_start[1] = 0;
  if (!p) return;
  const lmop_prefix* chain[2] = {p->parent ? p->parent : p, p->parent ? p : nullptr};
  for (int s = 0; s < 2; ++s)
    if (chain[s]) {
      r.seg_kv[s] = chain[s]->kv;
      r.seg_n[s] = chain[s]->n;
      r.seg_cap[s] = chain[s]->cap;
      r.seg_start[s] = chain[s]->slot0;
    }
}

void add_work(std::vector<int2>& work, int row, int n_q, int G) {
  const int tiles = attn_tiles(n_q, G);
  for (int t = 0; t < tiles; ++t) work.push_back(make_int2(row, t));
}

// Runs the constrained head over R rows whose final hidden states are at
// d_rowptr[i]; picks -> host.  dump_host (optional) receives [R][V] logits.
// Enqueues the head over R rows; the picks land in staging slot k (*picks),
// valid once the stream has passed this point.
lmop_status run_head(lmop_ctx* c, int k, int R, const std::vector<const float*>& rowptr,
                     const int32_t* d_sel, const int32_t* d_allowed, int n_sel, int n_allowed,
                     bool restricted, HeadPick** picks, float* dump_dev,
                     const uint8_t* d_state_mask = nullptr,
                     const std::vector<int32_t>* states = nullptr) {
  const lmop_config& cf = c->cfg;
  const int d = cf.d_model, V = cf.vocab;
  const int n_chunks = (V + kHeadVocabChunk - 1) / kHeadVocabChunk;
  const float** drp;
  uint16_t* hn;
  float2* part;
  float* zsel;
  HeadPick* dpk;
  LMOP_TRY(ws_get(c, "head_rowptr", R, &drp));
  LMOP_TRY(ws_get(c, "head_hn", (size_t)R * d, &hn));
  LMOP_TRY(ws_get(c, "head_part", restricted ? 1 : (size_t)R * n_chunks, &part));
  LMOP_TRY(ws_get(c, "head_zsel", (size_t)R * n_sel, &zsel));
  LMOP_TRY(ws_get(c, "head_pick", R, &dpk));
  const float** hrp;
  LMOP_TRY(stage_put(c, k, rowptr.data(), (size_t)R, &hrp));
  HIP_OK(c, hipMemcpyAsync(drp, hrp, R * sizeof(float*), hipMemcpyHostToDevice, c->stream));
  LMOP_TRY(timed(c, "rmsnorm_final", 0, (double)R * d * 6, [&] {
    return launch_rmsnorm(c->stream, nullptr, 0, drp, R, c->final_norm, d, cf.rms_eps, hn, d);
  }));
  if (restricted) {
    // only the allowed tokens' logits; the dump's other entries stay NaN
    if (dump_dev) HIP_OK(c, launch_fill_u32(c->stream, dump_dev, (size_t)R * V, 0xFFFFFFFFu));
    LMOP_TRY(timed(c, "head_restricted", 2.0 * R * n_sel * d,
                   (double)R * d * 2 + (double)n_sel * d * 2 + (double)R * n_sel * 4, [&] {
                     return launch_head_restricted(c->stream, hn, R, d, c->head, d_allowed, n_sel,
                                                   zsel, dump_dev, V);
                   }));
  } else {
    {
      GemmArgs ga{};
      ga.A = c->head;  // tiled
      ga.lda = d;
      ga.M = V;
      ga.N = R;
      ga.K = d;
      ga.bh = hn;
      ga.ldb = d;
      ga.part = part;
      ga.sel = d_sel;
      ga.zsel = zsel;
      ga.n_sel = n_sel;
      ga.dump = dump_dev;
      ga.ld_dump = V;
      LMOP_TRY(timed(c, "head_gemm", 2.0 * R * V * d, (double)V * d * 2 + (double)R * d * 2, [&] {
        return launch_gemm_f16(c->stream, ga, EPI_HEAD);
      }));
    }
  }
  // per-row automaton states: row r picks within state_mask[states[r]]
  int32_t* d_states = nullptr;
  if (states) {
    int32_t* hst;
    LMOP_TRY(ws_get(c, "head_state", R, &d_states));
    LMOP_TRY(stage_put(c, k, states->data(), (size_t)R, &hst));
    HIP_OK(c, hipMemcpyAsync(d_states, hst, R * sizeof(int32_t), hipMemcpyHostToDevice,
                             c->stream));
  }
  LMOP_TRY(timed(c, "head_finalize", 0, 0, [&] {
    return launch_head_finalize(c->stream, part, restricted ? 0 : n_chunks, zsel, n_sel,
                                n_allowed, d_allowed, R, dpk, d_states,
                                states ? d_state_mask : nullptr);
  }));
  LMOP_TRY(stage_put(c, k, (const HeadPick*)nullptr, (size_t)R, picks));
  HIP_OK(c, hipMemcpyAsync(*picks, dpk, R * sizeof(HeadPick), hipMemcpyDeviceToHost, c->stream));
  return LMOP_OK;
}

// Runs f with every scratch buffer carved from [base, base + bytes) (carve
// false: library-allocated scratch); no_alloc also forbids device, pinned and
// event allocations for the duration.
template <typename F>
lmop_status with_scratch(lmop_ctx* ctx, bool carve, char* base, size_t bytes, bool no_alloc,
                         F&& f) {
  ctx->carving = carve;
  ctx->carve_base = carve ? base : nullptr;
  ctx->carve_size = carve ? bytes : 0;
  ctx->no_alloc = no_alloc;
  const lmop_status st = f();
  // on any error, let the work already queued finish before returning, so
  // that none of it still reads or writes the caller's buffers or workspace
  if (st != LMOP_OK && !ctx->host_only && ctx->stream) (void)hipStreamSynchronize(ctx->stream);
  ctx->carving = false;
  ctx->carve_base = nullptr;
  ctx->carve_size = 0;
  ctx->no_alloc = false;
  ctx->carved.clear();
  return st;
}

}  // namespace

// ====================================================================== ABI
extern "C" {

const char* lmop_status_string(lmop_status s) {
  switch (s) {
    case LMOP_OK: return "ok";
    case LMOP_ERR_INVALID_ARG: return "invalid argument";
    case LMOP_ERR_STATE: return "call out of order";
    case LMOP_ERR_OOM: return "out of memory";
    case LMOP_ERR_DEVICE: return "device error";
    case LMOP_ERR_UNSUPPORTED: return "unsupported";
  }
  return "unknown status";
}


static thread_local std::string g_create_error;

// Device address of the static scratch array on each device, looked up once
// per device with that device current.
static std::mutex g_scratch_mu;
static std::map<int, void*> g_scratch_ptr;

static lmop_status bind_static_scratch(lmop_ctx* c) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  auto it = g_scratch_ptr.find(c->device);
  if (it == g_scratch_ptr.end()) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || ptr == nullptr) {
      (void)hipGetLastError();
      return fail(c, LMOP_ERR_DEVICE, "hipGetSymbolAddress of the scratch array failed: %s",
                  hipGetErrorString(e));
    }
    it = g_scratch_ptr.emplace(c->device, ptr).first;
  }
  c->static_scratch = it->second;
  return LMOP_OK;
}

lmop_status lmop_create(const lmop_config* cfg, int32_t device, void* hip_stream, lmop_ctx** out) {
  g_create_error.clear();
  if (!out) return LMOP_ERR_INVALID_ARG;
  *out = nullptr;
  std::unique_ptr<lmop_ctx> c(new lmop_ctx());
  lmop_ctx* cp = c.get();
  auto bail = [&](lmop_status st) {
    g_create_error = cp->err;
    if (!cp->host_only) {
      (void)dev_free(cp, cp->rope_tab);
      for (auto& stg : cp->stage)
        if (stg.done) (void)hipEventDestroy(stg.done);
      if (cp->own_stream && cp->stream) (void)hipStreamDestroy(cp->stream);
    }
    return st;
  };
  lmop_status st = check_config(cfg, cp);
  if (st != LMOP_OK) return bail(st);
  c->cfg = *cfg;
  if (c->cfg.max_seq == 0) c->cfg.max_seq = 4096;
  const lmop_config& cf = c->cfg;
  c->nq_dim = cf.n_heads * cf.head_dim;
  c->nkv_dim = cf.n_kv_heads * cf.head_dim;
  c->qkv_n = c->nq_dim + 2 * c->nkv_dim;
  c->f64 = round_up(cf.d_ff, 64);
  c->device = device;
  if (const char* inj = getenv("LMOP_INJECT_LAUNCH_FAILURE")) {
    const char* colon = strrchr(inj, ':');
    if (colon && colon != inj) {
      c->inject_name.assign(inj, colon - inj);
      c->inject_at = atol(colon + 1);
    }
  }
  if (device < 0) {
    c->host_only = true;
    *out = c.release();
    return LMOP_OK;
  }
  int n_dev = 0;
  if (hipGetDeviceCount(&n_dev) != hipSuccess || device >= n_dev) {
    (void)hipGetLastError();
    c->host_only = true;  // nothing to free on a device
    return bail(fail(cp, LMOP_ERR_DEVICE, "HIP device %d not available (%d devices)", device,
                     n_dev));
  }
  if (hipSetDevice(device) != hipSuccess)
    return bail(fail(cp, LMOP_ERR_DEVICE, "hipSetDevice(%d) failed", device));
  if (hip_stream) {
    c->stream = (hipStream_t)hip_stream;
  } else {
    // a blocking stream: work the caller queued on the null stream (torch's
    // default stream) completes before the library's work starts
    if (hipStreamCreateWithFlags(&c->stream, hipStreamDefault) != hipSuccess)
      return bail(fail(cp, LMOP_ERR_DEVICE, "hipStreamCreate failed"));
    c->own_stream = true;
  }
  st = bind_static_scratch(cp);
  if (st != LMOP_OK) return bail(st);
  // the staging slots' events exist before any call, so that a
  // no-allocation call creates none
  for (auto& stg : c->stage)
    if (hipEventCreateWithFlags(&stg.done, hipEventDisableTiming) != hipSuccess)
      return bail(fail(cp, LMOP_ERR_DEVICE, "hipEventCreate failed"));
  // rotary table: cos/sin of pos * theta^(-2i/hd) in double, stored fp32
  const int half = cf.head_dim / 2;
  std::vector<float2> tab((size_t)cf.max_seq * half);
  for (int p = 0; p < cf.max_seq; ++p)
    for (int i = 0; i < half; ++i) {
      const double ang = (double)p * std::pow((double)cf.rope_theta, -2.0 * i / cf.head_dim);
      tab[(size_t)p * half + i] = make_float2((float)std::cos(ang), (float)std::sin(ang));
    }
  void* rt = nullptr;
  st = dev_alloc(cp, &rt, tab.size() * sizeof(float2));
  if (st != LMOP_OK) return bail(st);
  c->rope_tab = (float2*)rt;
  if (hipMemcpy(rt, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice) != hipSuccess)
    return bail(fail(cp, LMOP_ERR_DEVICE, "upload of the rotary table failed"));
  *out = c.release();
  return LMOP_OK;
}

const char* lmop_last_error(const lmop_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_create_error.c_str();
}

static void destroy_prefix_storage(lmop_prefix* p) {
  if (p->store && --p->store->refs == 0) {
    (void)dev_free(p->ctx, p->store->kv);
    (void)dev_free(p->ctx, p->store->hidden);
    delete p->store;
  }
  p->store = nullptr;
  p->kv = nullptr;
  p->hidden = nullptr;
}

void lmop_destroy(lmop_ctx* ctx) {
  if (!ctx) return;
  if (!ctx->host_only) {
    (void)hipSetDevice(ctx->device);
    if (ctx->stream) (void)hipStreamSynchronize(ctx->stream);
  }
  for (lmop_prefix* p : ctx->prefixes) {
    destroy_prefix_storage(p);
    delete p;
  }
  ctx->prefixes.clear();
  if (!ctx->host_only) {
    free_weights(ctx);
    for (auto& kv : ctx->ws) (void)dev_free(ctx, kv.second.first);
    (void)dev_free(ctx, ctx->rope_tab);
    for (auto& s : ctx->spans) {
      (void)hipEventDestroy(s.a);
      (void)hipEventDestroy(s.b);
    }
    for (hipEvent_t e : ctx->ev_free) (void)hipEventDestroy(e);
    for (auto& st : ctx->stage) {
      if (st.p) (void)hipHostFree(st.p);
      if (st.done) (void)hipEventDestroy(st.done);
    }
    if (ctx->own_stream && ctx->stream) (void)hipStreamDestroy(ctx->stream);
  }
  delete ctx;
}

static lmop_status enter(lmop_ctx* ctx) {
  if (!ctx) return LMOP_ERR_INVALID_ARG;
  if (ctx->dead)
    return fail(ctx, LMOP_ERR_DEVICE, "ctx is unusable after an earlier error (%s)",
                ctx->err.c_str());
  ctx->err.clear();
  if (!ctx->host_only) HIP_OK(ctx, hipSetDevice(ctx->device));
  return LMOP_OK;
}

static void release_all_prefixes(lmop_ctx* c) {
  for (lmop_prefix* p : c->prefixes) {
    destroy_prefix_storage(p);
    delete p;
  }
  c->prefixes.clear();
}

lmop_status lmop_load_weights(lmop_ctx* ctx, const lmop_weights* w) {
  LMOP_TRY(enter(ctx));
  const lmop_config& cf = ctx->cfg;
  if (!w) return fail(ctx, LMOP_ERR_INVALID_ARG, "weights is NULL");
  if (w->n_layers != cf.n_layers)
    return fail(ctx, LMOP_ERR_INVALID_ARG, "weights have %d layers, config %d", w->n_layers,
                cf.n_layers);
  if (!w->tok_embedding || !w->lm_head || !w->final_norm || (cf.n_layers > 0 && !w->layers))
    return fail(ctx, LMOP_ERR_INVALID_ARG, "NULL embedding, head, final norm or layer array");
  if (w->format != (int32_t)LMOP_W_INT4_G32 && w->format != (int32_t)LMOP_W_FP8_E4M3)
    return fail(ctx, LMOP_ERR_INVALID_ARG, "unknown weight format %d", w->format);
  const int d = cf.d_model, nq = ctx->nq_dim, nkv = ctx->nkv_dim, F = cf.d_ff;
  for (int l = 0; l < cf.n_layers; ++l) {
    const lmop_layer& L = w->layers[l];
    if (!L.attn_norm || !L.mlp_norm)
      return fail(ctx, LMOP_ERR_INVALID_ARG, "layer %d: NULL norm gain", l);
    LMOP_TRY(check_qmat(ctx, "wq", l, L.wq, nq, d));
    LMOP_TRY(check_qmat(ctx, "wk", l, L.wk, nkv, d));
    LMOP_TRY(check_qmat(ctx, "wv", l, L.wv, nkv, d));
    LMOP_TRY(check_qmat(ctx, "wo", l, L.wo, d, nq));
    LMOP_TRY(check_qmat(ctx, "w_gate", l, L.w_gate, F, d));
    LMOP_TRY(check_qmat(ctx, "w_up", l, L.w_up, F, d));
    LMOP_TRY(check_qmat(ctx, "w_down", l, L.w_down, d, F));
  }
  if (ctx->host_only) {
    release_all_prefixes(ctx);
    ctx->generation++;
    ctx->loaded = true;
    return LMOP_OK;
  }
  HIP_OK(ctx, hipStreamSynchronize(ctx->stream));
  release_all_prefixes(ctx);
  free_weights(ctx);
  ctx->loaded = false;
  ctx->generation++;
  const bool od = w->on_device != 0;
  ctx->wfmt = (uint32_t)w->format;
  const size_t V = cf.vocab;
  void* p = nullptr;
  LMOP_TRY(upload(ctx, w->tok_embedding, V * d * 2, od, &p));
  ctx->emb = (uint16_t*)p;
  {  // the LM head, repacked into its tiles
    const void* src = w->lm_head;
    void* staged = nullptr;
    if (!od) {
      LMOP_TRY(dev_alloc(ctx, &staged, V * d * 2));
      HIP_OK(ctx, hipMemcpyAsync(staged, w->lm_head, V * d * 2, hipMemcpyHostToDevice,
                                 ctx->stream));
      src = staged;
    }
    const size_t vp = (V + kHeadTileRows - 1) / kHeadTileRows * kHeadTileRows;
    LMOP_TRY(dev_alloc(ctx, &p, vp * d * 2));
    ctx->weight_allocs.push_back(p);
    ctx->head = (uint16_t*)p;
    LMOP_TRY(timed(ctx, "repack_head", 0, 0, [&] {
      return launch_repack_head(ctx->stream, (const half_bits*)src, (int)V, d, ctx->head);
    }));
    if (staged) {
      HIP_OK(ctx, hipStreamSynchronize(ctx->stream));
      HIP_OK(ctx, dev_free(ctx, staged));
    }
  }
  LMOP_TRY(upload(ctx, w->final_norm, (size_t)d * 4, od, &p));
  ctx->final_norm = (float*)p;
  ctx->layers.resize(cf.n_layers);
  for (int l = 0; l < cf.n_layers; ++l) {
    const lmop_layer& L = w->layers[l];
    LayerW& D = ctx->layers[l];
    LMOP_TRY(upload(ctx, L.attn_norm, (size_t)d * 4, od, &p));
    D.attn_norm = (float*)p;
    LMOP_TRY(upload(ctx, L.mlp_norm, (size_t)d * 4, od, &p));
    D.mlp_norm = (float*)p;
    {  // fused q | k | v; q and k columns ordered so rotation pairs share a lane
      const lmop_qmat* s[3] = {&L.wq, &L.wk, &L.wv};
      std::vector<int32_t> m(round_up(ctx->qkv_n, 256), -1);
      const int hd = cf.head_dim, half = hd / 2, bph = hd / 64;
      int j = 0;
      for (int sec = 0; sec < 3; ++sec) {
        const int heads = sec == 0 ? cf.n_heads : cf.n_kv_heads;
        for (int h = 0; h < heads; ++h)
          for (int sub = 0; sub < bph; ++sub)
            for (int w = 0; w < 64; ++w, ++j) {
              const int f = w / 16, e = w % 16;
              const int dim = sec == 2 ? 64 * sub + w
                                       : (f < 2 ? 32 * sub + 16 * f + e
                                                : half + 32 * sub + 16 * (f - 2) + e);
              m[j] = (sec << 24) | (h * hd + dim);
            }
      }
      LMOP_TRY(pack(ctx, s, 3, m, ctx->qkv_n, d, od, &D.qkv));
    }
    {
      const lmop_qmat* s[1] = {&L.wo};
      const int rows[1] = {d};
      LMOP_TRY(pack(ctx, s, 1, concat_map(rows, 1, round_up(d, 256)), d, nq, od, &D.o));
    }
    {  // gate/up interleaved in blocks of 32: block b = [gate 32b..32b+31 | up 32b..32b+31]
      const lmop_qmat* s[2] = {&L.w_gate, &L.w_up};
      const int nblk = round_up(F, 32) / 32;
      std::vector<int32_t> m(round_up(nblk * 64, 256), -1);
      for (int b = 0; b < nblk; ++b)
        for (int i = 0; i < 32; ++i) {
          const int r = b * 32 + i;
          if (r < F) {
            m[b * 64 + i] = (0 << 24) | r;
            m[b * 64 + 32 + i] = (1 << 24) | r;
          }
        }
      LMOP_TRY(pack(ctx, s, 2, m, 2 * F, d, od, &D.gu));
    }
    {
      const lmop_qmat* s[1] = {&L.w_down};
      const int rows[1] = {d};
      LMOP_TRY(pack(ctx, s, 1, concat_map(rows, 1, round_up(d, 256)), d, F, od, &D.down));
    }
  }
  LMOP_TRY(sync(ctx));
  ctx->loaded = true;
  return LMOP_OK;
}

int32_t lmop_prefix_length(const lmop_prefix* p) { return p ? p->start + p->n : -1; }

// n prefixes of `parent`, prefix i = tokens[offsets[i] .. offsets[i+1]), all in
// one KV store: prefix i's slots start at slot0[i] (8-aligned), and the store
// is wide enough for every prefix's last 64-key attention block.  The
// forward passes are the batched prefill of row evaluation, so each prefix
// is bit for bit what a store of its own would hold.
static lmop_status make_prefixes(lmop_ctx* ctx, const lmop_prefix* parent, const int32_t* tokens,
                                 const int64_t* offsets, int n, lmop_prefix** out) {
  const lmop_config& cf = ctx->cfg;
  const int start = prefix_total(parent);
  std::vector<int> len(n), slot0(n);
  int64_t used = 0, need = 0;
  for (int i = 0; i < n; ++i) {
    len[i] = (int)(offsets[i + 1] - offsets[i]);
    slot0[i] = (int)std::min<int64_t>(used, kMaxStoreSlots);
    need = std::max<int64_t>(need, used + round_up(len[i], 64));
    used = round_up64(used + len[i], 8);
  }
  if (need > kMaxStoreSlots)
    return fail(ctx, LMOP_ERR_UNSUPPORTED,
                "%d prefixes of %lld tokens in all need more than %d KV slots: use several calls",
                n, (long long)offsets[n], kMaxStoreSlots);
  const int cap = round_up((int)need, 64);
  KvStore* store = nullptr;
  if (!ctx->host_only) {
    store = new KvStore();
    auto fail_free = [&](lmop_status st) {
      // work already queued may still write the store
      (void)hipStreamSynchronize(ctx->stream);
      (void)dev_free(ctx, store->kv);
      (void)dev_free(ctx, store->hidden);
      delete store;
      return st;
    };
    void* kv = nullptr;
    void* hid = nullptr;
    const size_t kv_bytes = (size_t)cf.n_layers * 2 * cap * ctx->nkv_dim * 2;
    lmop_status st = dev_alloc(ctx, &kv, kv_bytes);
    if (st != LMOP_OK) return fail_free(st);
    store->kv = (uint16_t*)kv;
    st = dev_alloc(ctx, &hid, (size_t)n * cf.d_model * 4);
    if (st != LMOP_OK) return fail_free(st);
    store->hidden = (float*)hid;
    // slots no prefix uses are read (masked) by attention: keep them finite
    if (launch_fill_u32(ctx->stream, kv, kv_bytes / 4, 0u) != hipSuccess)
      return fail_free(fail(ctx, LMOP_ERR_DEVICE, "clearing a prefix KV store failed"));
    const int G = cf.n_heads / cf.n_kv_heads;
    // prefixes in forward passes within the default token budget, or within
    // the largest budget whose scratch fits the carved region
    std::vector<std::pair<size_t, size_t>> passes;
    Need need;
    auto plan = [&](int b) {
      passes = make_batches(len, b);
      need = Need();
      batch_need(len, passes, G, &need);
      return !ctx->carving || scratch_total(ctx, need) <= ctx->carve_size;
    };
    if (ctx->carving) {
      if (fit_budget(kDefaultBatchTokens, plan) == 0)
        return fail_free(fail(ctx, LMOP_ERR_OOM,
                              "the workspace (%zu bytes) cannot hold the scratch of one prefix "
                              "pass (%zu bytes)",
                              ctx->carve_size, scratch_total(ctx, need)));
    } else {
      plan(kDefaultBatchTokens);
    }
    st = reserve_scratch(ctx, need);
    if (st != LMOP_OK) return fail_free(st);
    for (size_t pi = 0; pi < passes.size() && st == LMOP_OK; ++pi) {
      const int i0 = (int)passes[pi].first, i1 = (int)passes[pi].second;
      int T = 0;
      for (int i = i0; i < i1; ++i) T += len[i];
      const int R = i1 - i0;
      std::vector<int32_t> tok(T), pos(T), slot(T), last(R);
      std::vector<AttnRow> rows(R);
      std::vector<int2> work;
      Batch b;
      int t = 0;
      for (int i = i0; i < i1; ++i) {
        const int k = i - i0;
        for (int j = 0; j < len[i]; ++j) {
          tok[t + j] = tokens[offsets[i] + j];
          pos[t + j] = start + j;
          slot[t + j] = slot0[i] + j;
        }
        fill_segments(parent, rows[k]);
        rows[k].q_start = t;
        rows[k].n_q = len[i];
        rows[k].own_slot = slot0[i];
        rows[k].own_q0 = 0;
        add_work(work, k, len[i], G);
        last[k] = t + len[i] - 1;
        b.visible_keys += (double)len[i] * start + 0.5 * (double)len[i] * (len[i] + 1);
        t += len[i];
      }
      st = stage_begin(ctx, 0, stage_need(T, R, work.size()));
      if (st == LMOP_OK) st = upload_batch(ctx, 0, tok, pos, slot, rows, work, last);
      b.T = T;
      b.R = R;
      b.n_work = (int)work.size();
      b.own_kv = store->kv;
      b.own_cap = cap;
      b.n_last = cf.n_layers > 0 ? R : 0;
      if (st == LMOP_OK) st = forward(ctx, b);
      // the final hidden state of each prefix's last token (the whole model when L = 0)
      float* src = nullptr;
      if (st == LMOP_OK && cf.n_layers > 0) {
        st = ws_get(ctx, "xlast", (size_t)R * cf.d_model, &src);
        if (st == LMOP_OK &&
            hipMemcpyAsync(store->hidden + (size_t)i0 * cf.d_model, src,
                           (size_t)R * cf.d_model * 4, hipMemcpyDeviceToDevice,
                           ctx->stream) != hipSuccess)
          st = fail(ctx, LMOP_ERR_DEVICE, "copy of prefix hidden states failed");
      } else if (st == LMOP_OK) {
        st = ws_get(ctx, "x", (size_t)T * cf.d_model, &src);
        for (int k = 0; k < R && st == LMOP_OK; ++k)
          if (hipMemcpyAsync(store->hidden + (size_t)(i0 + k) * cf.d_model,
                             src + (size_t)last[k] * cf.d_model, (size_t)cf.d_model * 4,
                             hipMemcpyDeviceToDevice, ctx->stream) != hipSuccess)
            st = fail(ctx, LMOP_ERR_DEVICE, "copy of prefix hidden states failed");
      }
      if (st == LMOP_OK) st = stage_mark(ctx, 0);
      if (st == LMOP_OK) st = sync(ctx);
    }
    if (st != LMOP_OK) return fail_free(st);
    store->refs = n;
  }
  for (int i = 0; i < n; ++i) {
    lmop_prefix* p = new lmop_prefix();
    p->ctx = ctx;
    p->parent = const_cast<lmop_prefix*>(parent);
    p->n = len[i];
    p->start = start;
    p->cap = cap;
    p->slot0 = slot0[i];
    p->store = store;
    p->kv = store ? store->kv : nullptr;
    p->hidden = store ? store->hidden + (size_t)i * cf.d_model : nullptr;
    p->generation = ctx->generation;
    p->id = ctx->next_prefix_id++;
    ctx->prefixes.insert(p);
    out[i] = p;
  }
  if (parent) const_cast<lmop_prefix*>(parent)->children += n;
  return LMOP_OK;
}

// checks shared by lmop_set_prefix and lmop_set_prefixes
static lmop_status check_prefix_parent(lmop_ctx* ctx, const lmop_prefix* parent) {
  if (!ctx->loaded) return fail(ctx, LMOP_ERR_STATE, "lmop_load_weights has not succeeded");
  if (parent && !prefix_live(ctx, parent))
    return fail(ctx, LMOP_ERR_INVALID_ARG, "parent prefix is released or from another ctx");
  if (parent && parent->parent)
    return fail(ctx, LMOP_ERR_UNSUPPORTED, "a child prefix cannot have children");
  return LMOP_OK;
}

lmop_status lmop_set_prefix(lmop_ctx* ctx, const lmop_prefix* parent, const int32_t* tokens,
                            int32_t n_tokens, lmop_prefix** out) {
  if (out) *out = nullptr;
  LMOP_TRY(enter(ctx));
  if (!out) return fail(ctx, LMOP_ERR_INVALID_ARG, "out is NULL");
  LMOP_TRY(check_prefix_parent(ctx, parent));
  if (n_tokens < 1 || !tokens)
    return fail(ctx, LMOP_ERR_INVALID_ARG, "a prefix needs at least one token");
  LMOP_TRY(check_tokens(ctx, tokens, n_tokens, "prefix"));
  if (prefix_total(parent) + n_tokens >= ctx->cfg.max_seq)
    return fail(ctx, LMOP_ERR_INVALID_ARG, "prefix length %d exceeds max_seq %d",
                prefix_total(parent) + n_tokens, ctx->cfg.max_seq);
  const int64_t offs[2] = {0, n_tokens};
  return with_scratch(ctx, ctx->user_ws_bytes > 0, ctx->user_ws, ctx->user_ws_bytes, false,
                      [&] { return make_prefixes(ctx, parent, tokens, offs, 1, out); });
}

lmop_status lmop_set_prefixes(lmop_ctx* ctx, const lmop_prefix* parent, const int32_t* tokens,
                              const int64_t* offsets, int32_t n, lmop_prefix** out) {
  if (out && n > 0)
    for (int i = 0; i < n; ++i) out[i] = nullptr;
  LMOP_TRY(enter(ctx));
  if (n < 0) return fail(ctx, LMOP_ERR_INVALID_ARG, "n < 0");
  if (n == 0) return LMOP_OK;
  if (!out || !offsets || !tokens)
    return fail(ctx, LMOP_ERR_INVALID_ARG, "NULL tokens, offsets or out");
  LMOP_TRY(check_prefix_parent(ctx, parent));
  if (offsets[0] != 0) return fail(ctx, LMOP_ERR_INVALID_ARG, "offsets[0] != 0");
  for (int i = 0; i < n; ++i) {
    const int64_t len = offsets[i + 1] - offsets[i];
    if (len < 1) return fail(ctx, LMOP_ERR_INVALID_ARG, "prefix %d has no tokens", i);
    if (prefix_total(parent) + len >= ctx->cfg.max_seq)
      return fail(ctx, LMOP_ERR_INVALID_ARG, "prefix %d: length %lld exceeds max_seq %d", i,
                  (long long)(prefix_total(parent) + len), ctx->cfg.max_seq);
  }
  LMOP_TRY(check_tokens(ctx, tokens, offsets[n], "prefix"));
  return with_scratch(ctx, ctx->user_ws_bytes > 0, ctx->user_ws, ctx->user_ws_bytes, false,
                      [&] { return make_prefixes(ctx, parent, tokens, offsets, n, out); });
}

static void maybe_free_prefix(lmop_ctx* ctx, lmop_prefix* p) {
  while (p && p->released && p->children == 0) {
    lmop_prefix* par = p->parent;
    ctx->prefixes.erase(p);
    destroy_prefix_storage(p);
    delete p;
    if (par) par->children--;
    p = par;
  }
}

lmop_status lmop_release_prefix(lmop_ctx* ctx, lmop_prefix* prefix) {
  if (!ctx) return LMOP_ERR_INVALID_ARG;
  ctx->err.clear();
  if (!prefix || !ctx->prefixes.count(prefix) || prefix->released)
    return fail(ctx, LMOP_ERR_INVALID_ARG, "prefix is NULL, already released or from another ctx");
  if (!ctx->host_only && ctx->stream) {
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return fail(ctx, LMOP_ERR_DEVICE, "stream sync failed");
  }
  prefix->released = true;
  maybe_free_prefix(ctx, prefix);
  return LMOP_OK;
}

lmop_status lmop_dedup_rows(const int32_t* tokens, const int64_t* offsets, int32_t n_rows,
                            const int64_t* keys, int32_t* rep, int32_t* n_unique) {
  if (n_rows < 0 || !n_unique || (n_rows > 0 && (!offsets || !rep)))
    return LMOP_ERR_INVALID_ARG;
  if (n_rows == 0) {
    *n_unique = 0;
    return LMOP_OK;
  }
  if (offsets[0] != 0) return LMOP_ERR_INVALID_ARG;
  for (int r = 0; r < n_rows; ++r)
    if (offsets[r + 1] < offsets[r]) return LMOP_ERR_INVALID_ARG;
  if (offsets[n_rows] > 0 && !tokens) return LMOP_ERR_INVALID_ARG;
  dedup(tokens, offsets, n_rows, keys, rep, n_unique);
  return LMOP_OK;
}

// lmop_eval_rows with the scratch mode the ctx is in (library-allocated,
// carved from the caller's workspace, or carved from the static array)
static lmop_status eval_rows_impl(lmop_ctx* ctx, const lmop_prefix* prefix,
                                  const lmop_prefix* const* row_prefix, const int32_t* tokens,
                                  const int64_t* offsets, int32_t n_rows, const lmop_type* type,
                                  lmop_result* out, const lmop_eval_opts* opts) {
  if (!ctx->loaded) return fail(ctx, LMOP_ERR_STATE, "lmop_load_weights has not succeeded");
  if (n_rows < 0) return fail(ctx, LMOP_ERR_INVALID_ARG, "n_rows < 0");
  LMOP_TRY(check_type(ctx, type));
  if (n_rows == 0) return LMOP_OK;
  if (!offsets || (!out && !ctx->plan_out))
    return fail(ctx, LMOP_ERR_INVALID_ARG, "NULL offsets or out");
  if (offsets[0] != 0) return fail(ctx, LMOP_ERR_INVALID_ARG, "offsets[0] != 0");
  for (int r = 0; r < n_rows; ++r)
    if (offsets[r + 1] < offsets[r])
      return fail(ctx, LMOP_ERR_INVALID_ARG, "offsets decrease at row %d", r);
  const int64_t total = offsets[n_rows];
  if (total > 0 && !tokens) return fail(ctx, LMOP_ERR_INVALID_ARG, "tokens is NULL");
  LMOP_TRY(check_tokens(ctx, tokens, total, "row"));
  const lmop_config& cf = ctx->cfg;
  const bool is_aut = type->kind == LMOP_AUTOMATON;
  const int steps = type->kind == LMOP_INT || is_aut ? type->max_tokens : 1;
  const int dec = steps - 1;
  if (prefix && !prefix_live(ctx, prefix))
    return fail(ctx, LMOP_ERR_INVALID_ARG, "prefix is released or from another ctx");
  std::vector<const lmop_prefix*> pf(n_rows);
  for (int r = 0; r < n_rows; ++r) {
    const lmop_prefix* p = row_prefix ? row_prefix[r] : prefix;
    if (p && p != prefix && !prefix_live(ctx, p))
      return fail(ctx, LMOP_ERR_INVALID_ARG, "row %d: prefix is released or from another ctx", r);
    const int64_t len = offsets[r + 1] - offsets[r];
    if (!p && len == 0)
      return fail(ctx, LMOP_ERR_INVALID_ARG, "row %d has neither a prefix nor suffix tokens", r);
    if (prefix_total(p) + len + dec > cf.max_seq)
      return fail(ctx, LMOP_ERR_INVALID_ARG, "row %d: sequence of %lld tokens exceeds max_seq %d",
                  r, (long long)(prefix_total(p) + len + dec), cf.max_seq);
    pf[r] = p;
  }
  const uint32_t flags = opts ? opts->flags : 0u;
  if (flags & ~(LMOP_NO_DEDUP | LMOP_HEAD_RESTRICTED))
    return fail(ctx, LMOP_ERR_INVALID_ARG, "unknown flags 0x%x", (unsigned)flags);
  if (opts && opts->max_batch_tokens < 0)
    return fail(ctx, LMOP_ERR_INVALID_ARG, "max_batch_tokens < 0");
  const int limit = opts ? opts->limit : 0;
  const int64_t limit_value = opts ? opts->limit_value : 0;
  if (limit < 0) return fail(ctx, LMOP_ERR_INVALID_ARG, "limit < 0");

  const bool restricted = (flags & LMOP_HEAD_RESTRICTED) != 0;
  int budget = opts && opts->max_batch_tokens > 0 ? opts->max_batch_tokens : kDefaultBatchTokens;
  budget = std::min(budget, kMaxBatchBudget);
  float* dbg = opts ? opts->debug_logits : nullptr;
  const int V = cf.vocab;

  // early deduplication: one evaluation per distinct (prefix, suffix); a
  // row the mask leaves out gets a key of its own, so it represents no
  // other row, and is not evaluated
  const uint8_t* row_mask = opts ? opts->row_mask : nullptr;
  std::vector<int32_t> rep(n_rows);
  int32_t n_unique = 0;
  if (flags & LMOP_NO_DEDUP) {
    for (int r = 0; r < n_rows; ++r) rep[r] = r;
    n_unique = n_rows;
  } else {
    std::vector<int64_t> keys(n_rows);
    for (int r = 0; r < n_rows; ++r)
      keys[r] = row_mask && !row_mask[r] ? INT64_MIN + r : (pf[r] ? pf[r]->id : 0);
    dedup(tokens, offsets, n_rows, keys.data(), rep.data(), &n_unique);
  }
  std::vector<int32_t> uniq;
  uniq.reserve(n_unique);
  for (int r = 0; r < n_rows; ++r)
    if (rep[r] == r && (!row_mask || row_mask[r])) uniq.push_back(r);
  // group rows of one prefix together (attention reads that prefix's KV);
  // with a limit the rows stay in table order
  if (limit == 0)
    std::stable_sort(uniq.begin(), uniq.end(), [&](int a, int b) {
      const int64_t ia = pf[a] ? pf[a]->id : 0, ib = pf[b] ? pf[b]->id : 0;
      return ia < ib;
    });

  // allowed-token map: sel[token] = position in the allowed list (INT: EOS
  // last).  An automaton's list is every edge token in order of first
  // appearance, then EOS; each state allows a subset of it (a row of the
  // state mask table), and the head picks within the row's state's subset.
  const lmop_automaton* aut = type->automaton;
  std::vector<int32_t> allowed;
  std::vector<int32_t> sel(V, -1);
  if (is_aut) {
    for (int e = 0; e < aut->edge_offset[aut->n_states]; ++e)
      if (sel[aut->edge_token[e]] < 0) {
        sel[aut->edge_token[e]] = (int)allowed.size();
        allowed.push_back(aut->edge_token[e]);
      }
    if (type->eos_token >= 0) allowed.push_back(type->eos_token);
  } else {
    allowed.assign(type->tokens, type->tokens + type->n_tokens);
    if (type->kind == LMOP_INT) allowed.push_back(type->eos_token);
  }
  const int n_sel = (int)allowed.size();
  const int n_allowed0 = is_aut ? n_sel : type->n_tokens;
  for (int i = 0; i < n_sel; ++i) sel[allowed[i]] = i;
  std::vector<uint8_t> state_mask;
  if (is_aut) {
    const int S = aut->n_states;
    state_mask.assign((size_t)S * n_sel, 0);
    for (int st = 0; st < S; ++st) {
      for (int e = aut->edge_offset[st]; e < aut->edge_offset[st + 1]; ++e)
        state_mask[(size_t)st * n_sel + sel[aut->edge_token[e]]] = 1;
      if (aut->accepting[st] && type->eos_token >= 0)
        state_mask[(size_t)st * n_sel + n_sel - 1] = 1;
    }
  }

  const int G = cf.n_heads / cf.n_kv_heads;
  const int d = cf.d_model;
  std::vector<lmop_result> res(n_rows);
  // per distinct row (index into uniq): own tokens, slot of own token 0 in
  // its group's store, last chosen token
  std::vector<int> row_len(uniq.size()), own_slot(uniq.size());
  std::vector<int32_t> last_tok(uniq.size(), -1);
  std::vector<int32_t> row_state(uniq.size(), 0);  // automaton state
  for (size_t u = 0; u < uniq.size(); ++u)
    row_len[u] = (int)(offsets[uniq[u] + 1] - offsets[uniq[u]]);

  // The plan: batches within the token budget, decode groups, scratch sizes.
  // Library-allocated scratch takes the requested budget and decode groups
  // of at most kDecodeGroupBytes (and half the free memory); carved scratch
  // takes the largest budget whose plan fits, the own-KV store getting what
  // the other buffers leave.
  const size_t slot_bytes = (size_t)cf.n_layers * 2 * ctx->nkv_dim * 2;
  const int tiles1 = attn_tiles(1, G);
  Schedule sch;
  auto plan = [&](int b, size_t group_bytes) {
    sch = Schedule();
    sch.budget = b;
    sch.batches = make_batches(row_len, b);
    Need& n = sch.need;
    batch_need(row_len, sch.batches, G, &n);
    n.head_rows = n.R;
    n.restricted = restricted;
    n.dump = dbg != nullptr;
    n.n_sel = (size_t)n_sel;
    n.state_mask = state_mask.size();
    if (dec > 0) {
      // a decode step over every live row of a group: at most the group's rows
      const size_t ub = std::max(n.R, std::min((size_t)b, uniq.size()));
      Need other = n;
      other.T = std::max(other.T, ub);
      other.R = other.head_rows = std::max(other.R, ub);
      other.W = std::max(other.W, ub * tiles1);
      if (ctx->carving) {
        const size_t rest = scratch_total(ctx, other);
        if (rest + 256 >= ctx->carve_size) return false;
        group_bytes = ctx->carve_size - rest - 256;
      }
    }
    make_groups(row_len, dec, b, slot_bytes, group_bytes, &sch);
    size_t kv_slots = 0;
    for (size_t g = 0; g < sch.group_cap.size(); ++g) {
      kv_slots = std::max(kv_slots, (size_t)sch.group_cap[g]);
      if (dec > 0) {
        size_t rows = 0;
        for (size_t bi = 0; bi < sch.batches.size(); ++bi)
          if ((size_t)sch.group_of[bi] == g) rows += sch.batches[bi].second - sch.batches[bi].first;
        n.T = std::max(n.T, rows);
        n.R = std::max(n.R, rows);
        n.W = std::max(n.W, rows * tiles1);
        n.head_rows = std::max(n.head_rows, rows);
      }
    }
    n.own_kv = kv_slots * slot_bytes;
    return !ctx->carving || scratch_total(ctx, n) <= ctx->carve_size;
  };
  if (ctx->carving) {
    if (fit_budget(budget, [&](int b) { return plan(b, 0); }) == 0) {
      const int longest = row_len.empty() ? 0 : *std::max_element(row_len.begin(), row_len.end());
      return fail(ctx, LMOP_ERR_OOM,
                  "the %s (%zu bytes) cannot hold the scratch of one batch: a row of %d tokens "
                  "needs %zu bytes",
                  ctx->no_alloc ? "no-allocation scratch array" : "workspace", ctx->carve_size,
                  longest, scratch_total(ctx, sch.need));
    }
  } else {
    size_t group_bytes = kDecodeGroupBytes;
    if (dec > 0 && !ctx->host_only) {
      size_t free_b = 0, total_b = 0;
      if (hipMemGetInfo(&free_b, &total_b) == hipSuccess)
        group_bytes = std::max<size_t>(std::min(group_bytes, free_b / 2), 1);
    }
    plan(budget, group_bytes);
  }
  if (ctx->plan_out) {
    lmop_eval_plan& pl = *ctx->plan_out;
    pl.unique_rows = (int32_t)uniq.size();
    pl.batches = (int32_t)sch.batches.size();
    pl.batch_tokens = sch.budget;
    for (auto& bt : sch.batches) {
      int t = 0;
      for (size_t u = bt.first; u < bt.second; ++u) t += row_len[u];
      pl.max_batch_tokens = std::max(pl.max_batch_tokens, t);
    }
    pl.decode_groups = (int32_t)sch.group_cap.size();
    pl.scratch_bytes = scratch_total(ctx, sch.need);
    pl.own_kv_bytes = sch.need.own_kv;
    // the smallest workspace whose carved plan fits: a bisection over sizes
    // (a larger workspace never fits fewer rows), to the byte
    const bool was_carving = ctx->carving;
    const size_t was_size = ctx->carve_size;
    ctx->carving = true;
    auto fits = [&](size_t W) {
      ctx->carve_size = W;
      return fit_budget(budget, [&](int b) { return plan(b, 0); }) != 0;
    };
    size_t hi = std::max<size_t>((size_t)pl.scratch_bytes, (size_t)1 << 20);
    while (!fits(hi) && hi < ((size_t)1 << 50)) hi *= 2;
    size_t lo = 0;
    while (hi - lo > 1) {
      const size_t mid = lo + (hi - lo) / 2;
      (fits(mid) ? hi : lo) = mid;
    }
    pl.min_workspace_bytes = hi;
    ctx->carving = was_carving;
    ctx->carve_size = was_size;
    return LMOP_OK;
  }
  if (ctx->host_only)
    return fail(ctx, LMOP_ERR_UNSUPPORTED,
                "host-only ctx: arguments are valid and the plan fits (%zu batches, %zu bytes of "
                "scratch), no device to run",
                sch.batches.size(), scratch_total(ctx, sch.need));
  LMOP_TRY(reserve_scratch(ctx, sch.need));
  const auto& batches = sch.batches;
  const auto& base_of = sch.base_of;
  const auto& group_of = sch.group_of;
  const auto& group_cap = sch.group_cap;
  budget = sch.budget;

  int32_t *d_sel, *d_allowed;
  LMOP_TRY(ws_get(ctx, "sel", V, &d_sel));
  LMOP_TRY(ws_get(ctx, "allowed", n_sel, &d_allowed));
  HIP_OK(ctx, hipMemcpyAsync(d_sel, sel.data(), V * 4, hipMemcpyHostToDevice, ctx->stream));
  HIP_OK(ctx, hipMemcpyAsync(d_allowed, allowed.data(), n_sel * 4, hipMemcpyHostToDevice,
                             ctx->stream));
  uint8_t* d_state_mask = nullptr;
  if (is_aut) {
    LMOP_TRY(ws_get(ctx, "state_mask", state_mask.size(), &d_state_mask));
    HIP_OK(ctx, hipMemcpyAsync(d_state_mask, state_mask.data(), state_mask.size(),
                               hipMemcpyHostToDevice, ctx->stream));
  }
  HIP_OK(ctx, hipStreamSynchronize(ctx->stream));
  const int n_batches = (int)batches.size();

  // A batch between enqueue and collect: where its first step's picks land.
  struct InFlight {
    size_t u0 = 0;
    int R = 0;
    int k = 0;  // staging slot
    HeadPick* picks = nullptr;
    float* dump = nullptr;
  };
  uint16_t* own_kv = nullptr;  // the current group's store

  // Packs and uploads one batch, runs its prefill and its first head step;
  // nothing here waits for the GPU.
  auto enqueue = [&](int bi, InFlight& B) -> lmop_status {
    const size_t u0 = batches[bi].first, u1 = batches[bi].second;
    const int R = (int)(u1 - u0), k = bi & 1;
    const int cap_g = group_cap[group_of[bi]];
    if (bi == 0 || group_of[bi] != group_of[bi - 1])
      LMOP_TRY(ws_get(ctx, "own_kv", (size_t)cap_g * slot_bytes / 2, &own_kv, true));
    int T = 0;
    for (size_t u = u0; u < u1; ++u) T += row_len[u];
    std::vector<int32_t> tok(T), pos(T), slot(T);
    std::vector<AttnRow> rows(R);
    std::vector<int2> work;
    std::vector<int> qs(R);
    int t = 0, cap = base_of[bi];
    for (int i = 0; i < R; ++i) {
      const size_t u = u0 + i;
      const int r = uniq[u];
      const lmop_prefix* p = pf[r];
      const int len = row_len[u];
      own_slot[u] = cap;
      qs[i] = t;
      const int P = prefix_total(p);
      for (int j = 0; j < len; ++j) {
        tok[t + j] = tokens[offsets[r] + j];
        pos[t + j] = P + j;
        slot[t + j] = cap + j;
      }
      AttnRow& ar = rows[i];
      fill_segments(p, ar);
      ar.q_start = t;
      ar.n_q = len;
      ar.own_slot = cap;
      ar.own_q0 = 0;
      add_work(work, i, len, G);
      t += len;
      cap = round_up(cap + len + dec, 8);
    }
    // each row's last token (rows with suffix tokens only)
    std::vector<int32_t> last;
    std::vector<int> last_of(R, -1);
    for (int i = 0; i < R; ++i)
      if (row_len[u0 + i] > 0) {
        last_of[i] = (int)last.size();
        last.push_back(qs[i] + row_len[u0 + i] - 1);
      }
    LMOP_TRY(stage_begin(ctx, k, stage_need(T, R, work.size())));
    LMOP_TRY(upload_batch(ctx, k, tok, pos, slot, rows, work, last));
    Batch b;
    b.T = T;
    b.R = R;
    b.n_work = (int)work.size();
    b.own_kv = own_kv;
    b.own_cap = cap_g;
    b.n_last = cf.n_layers > 0 ? (int)last.size() : 0;
    for (int i = 0; i < R; ++i)
      b.visible_keys += (double)row_len[u0 + i] * prefix_total(pf[uniq[u0 + i]]) +
                        0.5 * (double)row_len[u0 + i] * (row_len[u0 + i] + 1);
    LMOP_TRY(forward(ctx, b));
    float* x;
    if (b.n_last > 0)
      LMOP_TRY(ws_get(ctx, "xlast", (size_t)b.n_last * d, &x));
    else
      LMOP_TRY(ws_get(ctx, "x", (size_t)std::max(T, 1) * d, &x));
    std::vector<const float*> rowptr(R);
    for (int i = 0; i < R; ++i) {
      const int r = uniq[u0 + i];
      if (row_len[u0 + i] == 0)
        rowptr[i] = pf[r]->hidden;
      else
        rowptr[i] = x + (size_t)(b.n_last > 0 ? last_of[i] : qs[i] + row_len[u0 + i] - 1) * d;
    }
    B.dump = nullptr;
    if (dbg) LMOP_TRY(ws_get(ctx, "dump", (size_t)R * V, &B.dump));
    std::vector<int32_t> st0;
    if (is_aut) st0.assign(R, 0);
    LMOP_TRY(run_head(ctx, k, R, rowptr, d_sel, d_allowed, n_sel, n_allowed0, restricted, &B.picks,
                      B.dump, d_state_mask, is_aut ? &st0 : nullptr));
    LMOP_TRY(stage_mark(ctx, k));
    B.u0 = u0;
    B.R = R;
    B.k = k;
    return LMOP_OK;
  };

  // Adds one step's pick to a row's result; true if the row decodes further.
  auto apply_pick = [&](size_t u, const HeadPick& hp) {
    lmop_result& o = res[uniq[u]];
    o.logprob += hp.logprob;
    o.logprob_full += hp.logprob_full;
    o.tokens[o.n_tokens++] = hp.token;
    if (is_aut) {
      // EOS ends the output in the current (accepting) state
      int32_t& st = row_state[u];
      if (type->eos_token >= 0 && hp.index == n_sel - 1) {
        o.value = st;
        return false;
      }
      int nxt = -1;
      for (int e = aut->edge_offset[st]; e < aut->edge_offset[st + 1]; ++e)
        if (aut->edge_token[e] == hp.token) nxt = aut->edge_next[e];
      if (nxt < 0) {  // not reachable: the state mask allows only edge tokens
        o.value = -1;
        return false;
      }
      st = nxt;
      const bool leaf = aut->edge_offset[st + 1] == aut->edge_offset[st];
      if (leaf || o.n_tokens >= steps) {
        o.value = aut->accepting[st] ? st : -1;
        return false;
      }
      last_tok[u] = hp.token;
      return true;
    }
    if (type->kind != LMOP_INT) {
      o.value = hp.index;
      return false;
    }
    if (hp.index == n_allowed0) return false;  // EOS
    o.value = o.value * 10 + hp.index;
    last_tok[u] = hp.token;
    return o.n_tokens < steps;
  };

  // Waits for a batch's first step and takes its picks; rows that decode
  // further join the group's live list.
  std::vector<size_t> live;
  auto collect = [&](InFlight& B) -> lmop_status {
    HIP_OK(ctx, hipEventSynchronize(ctx->stage[B.k].done));
    ctx->stage[B.k].pending = false;
    for (int i = 0; i < B.R; ++i) {
      const size_t u = B.u0 + i;
      const int r = uniq[u];
      lmop_result& o = res[r];
      o.value = 0;
      o.logprob = 0.f;
      o.logprob_full = 0.f;
      o.n_tokens = 0;
      for (int q = 0; q < 8; ++q) o.tokens[q] = -1;
      if (dbg) {
        std::fill(dbg + (size_t)r * steps * V, dbg + (size_t)(r + 1) * steps * V, NAN);
        HIP_OK(ctx, hipMemcpy(dbg + (size_t)r * steps * V, B.dump + (size_t)i * V,
                              (size_t)V * 4, hipMemcpyDeviceToHost));
      }
      if (apply_pick(u, B.picks[i])) live.push_back(u);
    }
    return LMOP_OK;
  };

  // The further (integer) steps of a group: one forward over all live rows
  // per step, each row adding one token to its own KV.
  auto decode = [&](int gi) -> lmop_status {
    for (int step = 1; step < steps && !live.empty(); ++step) {
      const int nl = (int)live.size();
      std::vector<int32_t> st(nl), sp(nl), ss(nl);
      std::vector<AttnRow> sr(nl);
      std::vector<int2> sw;
      for (int q = 0; q < nl; ++q) {
        const size_t u = live[q];
        const int r = uniq[u];
        const int own_idx = row_len[u] + step - 1;
        st[q] = last_tok[u];
        sp[q] = prefix_total(pf[r]) + own_idx;
        ss[q] = own_slot[u] + own_idx;
        fill_segments(pf[r], sr[q]);
        sr[q].q_start = q;
        sr[q].n_q = 1;
        sr[q].own_slot = own_slot[u];
        sr[q].own_q0 = own_idx;
        add_work(sw, q, 1, G);
      }
      LMOP_TRY(stage_begin(ctx, 0, stage_need(nl, nl, sw.size())));
      LMOP_TRY(upload_batch(ctx, 0, st, sp, ss, sr, sw));
      Batch sb;
      sb.T = nl;
      sb.R = nl;
      sb.n_work = (int)sw.size();
      sb.own_kv = own_kv;
      sb.own_cap = group_cap[gi];
      sb.decode = true;
      for (int q = 0; q < nl; ++q) sb.visible_keys += sp[q] + 1;  // position + 1 keys
      LMOP_TRY(forward(ctx, sb));
      float* x;
      LMOP_TRY(ws_get(ctx, "x", (size_t)nl * d, &x));
      std::vector<const float*> rowptr(nl);
      for (int q = 0; q < nl; ++q) rowptr[q] = x + (size_t)q * d;
      float* dump = nullptr;
      if (dbg) LMOP_TRY(ws_get(ctx, "dump", (size_t)nl * V, &dump));
      HeadPick* picks;
      std::vector<int32_t> st_live;
      if (is_aut)
        for (int q = 0; q < nl; ++q) st_live.push_back(row_state[live[q]]);
      LMOP_TRY(run_head(ctx, 0, nl, rowptr, d_sel, d_allowed, n_sel, n_sel, restricted, &picks,
                        dump, d_state_mask, is_aut ? &st_live : nullptr));
      LMOP_TRY(stage_mark(ctx, 0));
      HIP_OK(ctx, hipEventSynchronize(ctx->stage[0].done));
      ctx->stage[0].pending = false;
      std::vector<size_t> next;
      for (int q = 0; q < nl; ++q) {
        const size_t u = live[q];
        if (dbg)
          HIP_OK(ctx, hipMemcpy(dbg + ((size_t)uniq[u] * steps + step) * V,
                                dump + (size_t)q * V, (size_t)V * 4, hipMemcpyDeviceToHost));
        if (apply_pick(u, picks[q])) next.push_back(u);
      }
      live.swap(next);
    }
    live.clear();
    return LMOP_OK;
  };

  // Without a logit dump a batch's first step needs only its pinned picks:
  // the next batch of the same group (any next batch, for types without
  // further steps) is enqueued before this one is collected, so the GPU does
  // not wait while the host packs and reads back.  A logit dump reuses one
  // device buffer, so then each batch is collected before the next starts.
  // Early exit (limit > 0): once a batch (or a decode group) is final, every
  // table row before the first row not yet evaluated has its value; count
  // the qualifying ones in table order and stop at `limit`.
  std::vector<char> done(n_rows, 0);  // per representative row: evaluated
  int scan = 0, n_hits = 0;
  auto reached_limit = [&](size_t u_next) {
    const int upto = u_next < uniq.size() ? uniq[u_next] : n_rows;
    for (; scan < upto; ++scan)
      if (done[rep[scan]] && res[rep[scan]].value == limit_value) ++n_hits;
    return n_hits >= limit;
  };
  InFlight fl[2];
  int next_b = 0;
  for (int bi = 0; bi < n_batches; ++bi) {
    if (next_b == bi) LMOP_TRY(enqueue(next_b++, fl[bi & 1]));
    const bool last_of_group = bi + 1 == n_batches || group_of[bi + 1] != group_of[bi];
    if (!dbg && next_b == bi + 1 && bi + 1 < n_batches && (dec == 0 || !last_of_group))
      LMOP_TRY(enqueue(next_b++, fl[(bi + 1) & 1]));
    LMOP_TRY(collect(fl[bi & 1]));
    for (size_t u = batches[bi].first; u < batches[bi].second; ++u) done[uniq[u]] = 1;
    if (dec > 0 && last_of_group) LMOP_TRY(decode(group_of[bi]));
    if (limit > 0 && (dec == 0 || last_of_group) && reached_limit(batches[bi].second)) break;
  }
  LMOP_TRY(sync(ctx));
  lmop_result skipped;
  skipped.value = -1;
  skipped.logprob = skipped.logprob_full = NAN;
  skipped.n_tokens = 0;
  for (int q = 0; q < 8; ++q) skipped.tokens[q] = -1;
  for (int r = 0; r < n_rows; ++r) {
    if (!done[rep[r]]) {
      out[r] = skipped;
      if (dbg) std::fill(dbg + (size_t)r * steps * V, dbg + (size_t)(r + 1) * steps * V, NAN);
      continue;
    }
    out[r] = res[rep[r]];
    if (dbg && rep[r] != r)
      std::memcpy(dbg + (size_t)r * steps * V, dbg + (size_t)rep[r] * steps * V,
                  (size_t)steps * V * sizeof(float));
  }
  // a large library-allocated own-KV store is returned after the call
  if (!ctx->carving) {
    auto it = ctx->ws.find("own_kv");
    if (it != ctx->ws.end() && it->second.second > kKeepOwnKvBytes)
      LMOP_TRY(ws_release(ctx, "own_kv"));
  }
  return LMOP_OK;
}

lmop_status lmop_eval_rows(lmop_ctx* ctx, const lmop_prefix* prefix,
                           const lmop_prefix* const* row_prefix, const int32_t* tokens,
                           const int64_t* offsets, int32_t n_rows, const lmop_type* type,
                           lmop_result* out, const lmop_eval_opts* opts) {
  LMOP_TRY(enter(ctx));
  return with_scratch(ctx, ctx->user_ws_bytes > 0, ctx->user_ws, ctx->user_ws_bytes, false, [&] {
    return eval_rows_impl(ctx, prefix, row_prefix, tokens, offsets, n_rows, type, out, opts);
  });
}

lmop_status lmop_eval_rows_noalloc(lmop_ctx* ctx, const lmop_prefix* prefix,
                                   const lmop_prefix* const* row_prefix, const int32_t* tokens,
                                   const int64_t* offsets, int32_t n_rows, const lmop_type* type,
                                   lmop_result* out, const lmop_eval_opts* opts) {
  LMOP_TRY(enter(ctx));
  if (!ctx->host_only && !ctx->static_scratch)
    return fail(ctx, LMOP_ERR_STATE, "the static scratch array is not bound on device %d",
                ctx->device);
  return with_scratch(ctx, true, (char*)ctx->static_scratch, kNoAllocScratchBytes, true, [&] {
    return eval_rows_impl(ctx, prefix, row_prefix, tokens, offsets, n_rows, type, out, opts);
  });
}

lmop_status lmop_plan_rows(lmop_ctx* ctx, const lmop_prefix* prefix,
                           const lmop_prefix* const* row_prefix, const int32_t* tokens,
                           const int64_t* offsets, int32_t n_rows, const lmop_type* type,
                           const lmop_eval_opts* opts, lmop_eval_plan* plan) {
  LMOP_TRY(enter(ctx));
  if (!plan) return fail(ctx, LMOP_ERR_INVALID_ARG, "plan is NULL");
  *plan = lmop_eval_plan{};
  ctx->plan_out = plan;
  const lmop_status st =
      with_scratch(ctx, ctx->user_ws_bytes > 0, ctx->user_ws, ctx->user_ws_bytes, false, [&] {
        return eval_rows_impl(ctx, prefix, row_prefix, tokens, offsets, n_rows, type, nullptr,
                              opts);
      });
  ctx->plan_out = nullptr;
  return st;
}

lmop_status lmop_set_workspace(lmop_ctx* ctx, void* dev_ptr, size_t bytes) {
  LMOP_TRY(enter(ctx));
  if ((dev_ptr == nullptr) != (bytes == 0))
    return fail(ctx, LMOP_ERR_INVALID_ARG, "a workspace needs both a pointer and a size");
  if (((uintptr_t)dev_ptr & 255) != 0)
    return fail(ctx, LMOP_ERR_INVALID_ARG, "the workspace must be 256-byte aligned");
  if (dev_ptr && !ctx->host_only) {
    hipPointerAttribute_t at;
    if (hipPointerGetAttributes(&at, dev_ptr) != hipSuccess || at.type != hipMemoryTypeDevice ||
        at.device != ctx->device) {
      (void)hipGetLastError();
      return fail(ctx, LMOP_ERR_INVALID_ARG, "the workspace is not device memory of device %d",
                  ctx->device);
    }
  }
  if (!ctx->host_only) {
    // the previous workspace (or library scratch) may still be read
    HIP_OK(ctx, hipStreamSynchronize(ctx->stream));
    if (dev_ptr) LMOP_TRY(ws_release_all(ctx));
  }
  ctx->user_ws = (char*)dev_ptr;
  ctx->user_ws_bytes = bytes;
  ctx->user_ws_peak = 0;
  return LMOP_OK;
}

lmop_status lmop_get_memory(const lmop_ctx* ctx, lmop_memory_stats* out) {
  if (!ctx || !out) return LMOP_ERR_INVALID_ARG;
  out->device_bytes = ctx->dev_bytes;
  out->device_peak = ctx->dev_peak;
  out->workspace_bytes = ctx->user_ws_bytes;
  out->workspace_peak = ctx->user_ws_peak;
  return LMOP_OK;
}

lmop_status lmop_set_profiling(lmop_ctx* ctx, int32_t period) {
  if (!ctx) return LMOP_ERR_INVALID_ARG;
  if (period < 0) return fail(ctx, LMOP_ERR_INVALID_ARG, "profiling period %d < 0", period);
  if (!ctx->host_only) LMOP_TRY(sync(ctx));
  ctx->prof = period;
  ctx->stats.clear();
  return LMOP_OK;
}

lmop_status lmop_get_kernel_stats(lmop_ctx* ctx, lmop_kernel_stat* out, int32_t max_entries,
                                  int32_t* n_entries) {
  if (!ctx || !n_entries || max_entries < 0 || (max_entries > 0 && !out))
    return LMOP_ERR_INVALID_ARG;
  if (!ctx->host_only) LMOP_TRY(sync(ctx));
  int i = 0;
  for (auto& kv : ctx->stats) {
    if (i < max_entries) {
      lmop_kernel_stat& s = out[i];
      std::memset(&s, 0, sizeof s);
      std::snprintf(s.name, sizeof s.name, "%s", kv.first.c_str());
      s.launches = kv.second.launches;
      s.timed_launches = kv.second.timed;
      s.total_ms = kv.second.ms;
      s.flops = kv.second.flops;
      s.bytes = kv.second.bytes;
    }
    ++i;
  }
  *n_entries = i;
  return LMOP_OK;
}

}  // extern "C"
