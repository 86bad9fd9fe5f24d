// Host runtime behind include/atspeed.h: workspace layout, item trie, the
// decoder forward over planned rows, and the draft / verify / decode calls.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/atspeed.h"
#include "common.h"
#include "kernels.h"
#include "select.h"

using namespace atspeed;

namespace {

thread_local std::string g_err;

atspeed_status fail(atspeed_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

#define HIP_TRY(expr)                                                                      \
  do {                                                                                     \
    hipError_t _e = (expr);                                                                \
    if (_e != hipSuccess) return fail(ATSPEED_E_DEVICE, std::string(#expr) + ": " + hipGetErrorString(_e)); \
  } while (0)

#define ST_TRY(expr)                        \
  do {                                      \
    atspeed_status _s = (expr);             \
    if (_s != ATSPEED_OK) return _s;        \
  } while (0)

// Bump allocator over the caller's workspace (a null base only measures).
struct Arena {
  char* base;
  size_t off = 0;
  template <class T>
  T* take(size_t n) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
};

struct ModelRt {
  atspeed_model_dims dims{};
  bool present = false;
  const void* emb = nullptr;
  std::vector<const void*> layers;
  const float* final_norm = nullptr;
  const void* lm_head = nullptr;
  void* pk = nullptr;            // prefix cache [layers][B][H][Pmax][dh]
  void* pv = nullptr;
  void* tk = nullptr;            // tree KV [tree_layers][B*Tmax][d]
  void* tv = nullptr;
  size_t tkv_layer_stride = 0;   // elements between layers (0: one shared buffer)
  int kv_layer0 = 0;             // first tree-KV layer of the current buffer set (tree-KV reuse)
  size_t pkv_layer_stride = 0;
  float* cosT = nullptr;
  float* sinT = nullptr;
  float* ropeT = nullptr;
  float* lp = nullptr;           // [B*Tmax][nitem] log-probs by tree slot
  float* root = nullptr;         // [B][nitem] log-probs at the last prefix position
  int dh() const { return dims.d_model / dims.n_heads; }
};

struct HostTrie {
  std::vector<int> code, first, cnt;
  int child(int node, int c) const {
    int lo = first[node], hi = lo + cnt[node] - 1;
    while (lo <= hi) {
      int mid = (lo + hi) / 2;
      if (code[mid] == c) return mid;
      if (code[mid] < c) lo = mid + 1; else hi = mid - 1;
    }
    return -1;
  }
};

}  // namespace

struct atspeed_ctx {
  atspeed_config cfg{};
  hipStream_t st = nullptr;
  bool bf16 = false;
  int Tmax = 0, Mmax = 0, nitem = 0, max_cand = 0, max_pos = 0;
  ModelRt tgt, dft;
  HostTrie htrie;
  TrieDev trie{};
  StateDev state{};
  TreeDev tree{};
  Rows rows{};
  float* x = nullptr;
  void* xn = nullptr;
  void* q = nullptr;
  void* ao = nullptr;
  void* h = nullptr;
  float* logits = nullptr;
  float* scratch = nullptr;
  float* part = nullptr;      // bf16: second k-half of the o / down product [Mmax, d] fp32
  int* lo = nullptr;
  int* hi = nullptr;
  int* lvl_lo = nullptr;
  int* lvl_hi = nullptr;
  int* row_last = nullptr;
  int* Mb = nullptr;         // [1] = B (rows of the last-position head in prefill)
  int* Mall = nullptr;       // [1] = B * Tmax (every tree slot)
  int* plan_max = nullptr;   // [1] largest per-user row count of the last tree plan (scratch word)
  int shared_prefix = 0;     // prefix positions the users of the last prefill shared
  int* err = nullptr;
  int* acc_tmp = nullptr;
  int* tafter_tmp = nullptr;
  unsigned long long* keys = nullptr;
  CandBuf cand{};
  RelaxArgs relax{};
  int B = 0, P = 0;
  bool prefilled = false;
  bool drafted = false;
  // tree-KV reuse (cfg.reuse_tree_kv): the target's per-layer tree K/V and its
  // log-probs by slot live in two buffer sets that alternate between verifies;
  // a verify of the decode loop takes the nodes the previous one already
  // forwarded from the other set instead of forwarding them again
  bool reuse = false;
  int kv_cur = 0;               // set holding the last verify's K/V and log-probs
  bool carry_ok = false;        // the last verify was the decode loop's own, since the prefill
  float* lp_set[2] = {nullptr, nullptr};
  // device address of the static scratch of atspeed_accept_noalloc on the
  // context's device (taken at create)
  unsigned char* static_scratch = nullptr;
  // draft alignment
  void* root_h = nullptr;          // [B, d_draft] the draft's final-normed hidden state at each user's root
  int* align_kslot = nullptr;      // [B, L] slot of the last training sequence's depth-t prefix
  float* loss_rows = nullptr;      // [Mmax] weighted loss of each context row
  bool align_ready = false;        // the tree holds the contexts of the last atspeed_align_data
  bool dft_prefilled = false;      // the draft's prefix caches hold the last prefill's users
  uint32_t* prev_tpath = nullptr;  // [B*Tmax] path keys of the last verify's tree
  int* prev_depth = nullptr;       // [B*Tmax]
  int* prev_n = nullptr;           // [B] its forwarded (or carried) nodes: slots [0, prev_n)
  int* src = nullptr;              // [B*Tmax] previous slot of each node or -1
  int* fidx = nullptr;             // [B*Tmax] per user, the nodes still to forward
  int* fcnt = nullptr;             // [B]
  int64_t rows_fwd = 0;            // target tree rows forwarded (decode statistics)
  // residual-stream capture of the next target forward (atspeed_capture_hidden)
  float* cap_x = nullptr;        // [2 n_layers + 1][cap_rows][d] fp32
  bf16_t* cap_act = nullptr;     // bf16 inputs of every GEMM and attention (layout at atspeed_capture_hidden)
  int32_t* cap_plan = nullptr;   // [3][cap_rows] user, position, slot of each row; then the row count
  int cap_rows = 0;
  int cap_model = 0;             // 0 target, 1 draft
  int cap_skip = 0;              // forwards of that model to let pass before the captured one
  // timing instrumentation
  uint32_t timing_mask = 0;   // kernel classes whose launches are bracketed by events
  bool timing_target_only = false;  // skip the draft model's launches
  const ModelRt* fwd_model = nullptr;  // model of the forward being enqueued (null: none)
  std::vector<hipEvent_t> ev_pool;
  std::vector<int> ev_kind;   // kind of the interval that starts at event i (-1: end marker)
  std::vector<double> ev_flops;  // algorithmic flops of that interval's launch
  size_t ev_used = 0;
  double t_ms[ATSPEED_K_COUNT] = {};
  int64_t t_n[ATSPEED_K_COUNT] = {};
  double t_flop[ATSPEED_K_COUNT] = {};
  ~atspeed_ctx() {
    for (hipEvent_t e : ev_pool) hipEventDestroy(e);
  }
};

namespace {

size_t esize(const atspeed_ctx& c) { return c.bf16 ? 2 : 4; }

// Marks the start of a launch of class `kind` (or, with kind -1, the end of the
// previous one) when timing is on.
hipError_t mark(atspeed_ctx& c, int kind, double flops = 0.0) {
  if (!c.timing_mask) return hipSuccess;
  // An event opens a span before a launch of a selected class; the next mark
  // closes it (and opens a new span if its class is selected too).
  const bool draft = c.fwd_model != nullptr && c.fwd_model == &c.dft;
  const bool want = kind >= 0 && ((c.timing_mask >> kind) & 1u) && !(draft && c.timing_target_only);
  const bool open = c.ev_used > 0 && c.ev_kind[c.ev_used - 1] >= 0;
  if (!want && !open) return hipSuccess;
  if (c.ev_used == c.ev_pool.size()) {
    hipEvent_t e;
    hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) return err;
    c.ev_pool.push_back(e);
    c.ev_kind.push_back(-1);
    c.ev_flops.push_back(0.0);
  }
  c.ev_kind[c.ev_used] = want ? kind : -1;
  c.ev_flops[c.ev_used] = want && !draft ? flops : 0.0;
  return hipEventRecord(c.ev_pool[c.ev_used++], c.st);
}

hipError_t fold_timing(atspeed_ctx& c) {
  if (c.ev_used == 0) return hipSuccess;
  hipError_t err = hipEventSynchronize(c.ev_pool[c.ev_used - 1]);
  if (err != hipSuccess) return err;
  for (size_t i = 0; i + 1 < c.ev_used; ++i) {
    const int k = c.ev_kind[i];
    if (k < 0) continue;
    float ms = 0.f;
    err = hipEventElapsedTime(&ms, c.ev_pool[i], c.ev_pool[i + 1]);
    if (err != hipSuccess) return err;
    c.t_ms[k] += ms;
    c.t_n[k] += 1;
    c.t_flop[k] += c.ev_flops[i];
  }
  c.ev_used = 0;
  return hipSuccess;
}

#define MARK(kind) HIP_TRY(mark(c, kind))
#define MARK_F(kind, flops) HIP_TRY(mark(c, kind, flops))

atspeed_status check_dims(const atspeed_model_dims& m, const atspeed_config& c, const char* who) {
  std::string w(who);
  if (m.n_layers < 1 || m.d_model < 1 || m.n_heads < 1 || m.d_ffn < 1)
    return fail(ATSPEED_E_INVALID, w + ": non-positive dimension");
  if (m.d_model % m.n_heads) return fail(ATSPEED_E_SHAPE, w + ": d_model % n_heads != 0");
  int dh = m.d_model / m.n_heads;
  if (c.dtype == ATSPEED_BF16) {
    if (dh != 64 && dh != 128) return fail(ATSPEED_E_SHAPE, w + ": bf16 needs d_head 64 or 128");
    if (m.d_model % 256 || m.d_ffn % 128) return fail(ATSPEED_E_SHAPE, w + ": bf16 needs d_model % 256 == 0 and d_ffn % 128 == 0");
  } else {
    if (dh != 32 && dh != 64 && dh != 128) return fail(ATSPEED_E_SHAPE, w + ": d_head must be 32, 64 or 128");
    if (m.d_model % 16 || m.d_ffn % 16) return fail(ATSPEED_E_SHAPE, w + ": d_model, d_ffn must be multiples of 16");
  }
  if (m.d_model > 8192) return fail(ATSPEED_E_SHAPE, w + ": d_model above 8192 (row kernels hold a row in registers)");
  if (m.item_base < 0 || m.vocab < m.item_base + c.L * c.codebook)
    return fail(ATSPEED_E_SHAPE, w + ": vocab must hold item_base + L*codebook tokens");
  return ATSPEED_OK;
}

atspeed_status check_config(const atspeed_config* cfg) {
  if (!cfg) return fail(ATSPEED_E_INVALID, "config is null");
  const atspeed_config& c = *cfg;
  if (c.L < 1 || c.L > 4) return fail(ATSPEED_E_INVALID, "L must be 1..4");
  if (c.codebook < 1 || c.codebook > 256) return fail(ATSPEED_E_INVALID, "codebook must be 1..256");
  if (c.K < 1 || c.K > kMaxSel) return fail(ATSPEED_E_INVALID, "K must be 1..128");
  if (c.N < c.K || c.N > kMaxSel) return fail(ATSPEED_E_INVALID, "N must be K..128");
  if (c.gamma < 1) return fail(ATSPEED_E_INVALID, "gamma must be >= 1");
  if (c.sd_start_level != 0 && c.sd_start_level != 1) return fail(ATSPEED_E_INVALID, "sd_start_level must be 0 or 1");
  if (c.reuse_tree_kv != 0 && c.reuse_tree_kv != 1) return fail(ATSPEED_E_INVALID, "reuse_tree_kv must be 0 or 1");
  if (c.max_batch < 1 || c.max_batch > 1024) return fail(ATSPEED_E_INVALID, "max_batch must be 1..1024");
  if (c.max_prefix < 1) return fail(ATSPEED_E_INVALID, "max_prefix must be >= 1");
  if (c.dtype != ATSPEED_FP32 && c.dtype != ATSPEED_BF16) return fail(ATSPEED_E_INVALID, "dtype");
  if (c.mode != ATSPEED_STRICT && c.mode != ATSPEED_RELAXED_EXACT && c.mode != ATSPEED_RELAXED_PAPER)
    return fail(ATSPEED_E_INVALID, "mode must be strict, relaxed-exact or relaxed-paper");
  if (c.mode != ATSPEED_STRICT && !(c.temperature > 0.f)) return fail(ATSPEED_E_INVALID, "temperature must be > 0");
  if (c.mode != ATSPEED_STRICT && c.sd_start_level != 0)
    return fail(ATSPEED_E_INVALID, "sd_start_level 1 is defined for strict verification only");
  ST_TRY(check_dims(c.target, c, "target"));
  if (c.draft.n_layers > 0) {
    ST_TRY(check_dims(c.draft, c, "draft"));
    if (c.draft.item_base != c.target.item_base) return fail(ATSPEED_E_SHAPE, "draft and target item_base differ");
  }
  // Row offsets inside an activation matrix are 32-bit in the kernels: rows x
  // widest row must stay below 2^31 elements.
  const long long tmax = (long long)c.K * (c.L - 1) + (long long)c.gamma * c.N;
  const long long rows = (long long)c.max_batch * std::max<long long>(c.max_prefix, tmax);
  const long long width = std::max({c.target.d_model, c.target.d_ffn, c.draft.d_model, c.draft.d_ffn, 4 * c.codebook});
  if (rows * width >= (1LL << 31))
    return fail(ATSPEED_E_SHAPE, "max_batch x max(max_prefix, tree rows) x widest activation row must be below 2^31");
  return ATSPEED_OK;
}

atspeed_status build_trie(const atspeed_config& c, const atspeed_catalog* cat, HostTrie& t) {
  if (!cat || !cat->codes || cat->n_items < 1) return fail(ATSPEED_E_INVALID, "catalog is empty or null");
  if (cat->n_items < c.K) return fail(ATSPEED_E_INVALID, "catalog holds fewer than K items");
  std::vector<uint32_t> keys(cat->n_items);
  for (int i = 0; i < cat->n_items; ++i) {
    uint32_t k = 0;
    for (int l = 0; l < c.L; ++l) {
      int code = cat->codes[(size_t)i * c.L + l];
      if (code < 0 || code >= c.codebook) return fail(ATSPEED_E_INVALID, "catalog code out of range");
      k |= (uint32_t)code << (8 * (3 - l));
    }
    keys[i] = k;
  }
  std::sort(keys.begin(), keys.end());
  if (std::adjacent_find(keys.begin(), keys.end()) != keys.end()) return fail(ATSPEED_E_INVALID, "catalog has duplicate items");
  // level-ordered unique prefixes; node 0 = root
  std::vector<std::vector<uint32_t>> lv(c.L + 1);
  lv[0] = {0u};
  for (int l = 1; l <= c.L; ++l) {
    uint32_t mask = l == 4 ? 0xFFFFFFFFu : ~(0xFFFFFFFFu >> (8 * l));
    for (uint32_t k : keys) {
      uint32_t p = k & mask;
      if (lv[l].empty() || lv[l].back() != p) lv[l].push_back(p);
    }
  }
  std::vector<int> off(c.L + 2, 0);
  for (int l = 0; l <= c.L; ++l) off[l + 1] = off[l] + (int)lv[l].size();
  const int n = off[c.L + 1];
  t.code.assign(n, 0);
  t.first.assign(n, 0);
  t.cnt.assign(n, 0);
  for (int l = 1; l <= c.L; ++l) {
    uint32_t pmask = l == 1 ? 0u : ~(0xFFFFFFFFu >> (8 * (l - 1)));
    size_t pi = 0;
    for (size_t i = 0; i < lv[l].size(); ++i) {
      uint32_t p = lv[l][i];
      while ((lv[l - 1][pi] & pmask) != (p & pmask)) ++pi;
      int id = off[l] + (int)i, pid = off[l - 1] + (int)pi;
      t.code[id] = (p >> (8 * (3 - (l - 1)))) & 0xFF;
      if (t.cnt[pid] == 0) t.first[pid] = id;
      t.cnt[pid]++;
    }
  }
  return ATSPEED_OK;
}

// Lays out (base == null: measures) every device buffer of a context.
void layout(atspeed_ctx& c, const atspeed_config& cfg, int trie_nodes, Arena& a) {
  const int B = cfg.max_batch, P = cfg.max_prefix, L = cfg.L;
  c.bf16 = cfg.dtype == ATSPEED_BF16;
  c.nitem = L * cfg.codebook;
  c.Tmax = cfg.K * (L - 1) + cfg.gamma * cfg.N;
  c.Mmax = std::max(B * P, B * c.Tmax);
  c.max_cand = cfg.N * cfg.codebook;
  c.max_pos = P + L;
  const size_t es = c.bf16 ? 2 : 4;
  const int Tm = c.Tmax;
  c.trie.code = a.take<int>(trie_nodes);
  c.trie.first = a.take<int>(trie_nodes);
  c.trie.cnt = a.take<int>(trie_nodes);
  int dmax = cfg.target.d_model, fmax = cfg.target.d_ffn;
  ModelRt* ms[2] = {&c.tgt, &c.dft};
  const atspeed_model_dims* ds[2] = {&cfg.target, &cfg.draft};
  for (int w = 0; w < 2; ++w) {
    const atspeed_model_dims& m = *ds[w];
    ModelRt& r = *ms[w];
    r.dims = m;
    if (m.n_layers <= 0) continue;
    dmax = std::max(dmax, m.d_model);
    fmax = std::max(fmax, m.d_ffn);
    const size_t pkv = (size_t)m.n_layers * B * P * m.d_model;
    r.pkv_layer_stride = (size_t)B * P * m.d_model;
    r.pk = a.take<char>(pkv * es);
    r.pv = a.take<char>(pkv * es);
    // the target's tree K/V is dead once a layer's attention has run, so one
    // buffer serves every layer -- unless it is kept for the next verify
    const bool keep = w == 0 && cfg.reuse_tree_kv;
    const int tl = w == 0 ? (keep ? 2 * m.n_layers : 1) : m.n_layers;
    r.tkv_layer_stride = w == 0 && !keep ? 0 : (size_t)B * Tm * m.d_model;
    r.tk = a.take<char>((size_t)tl * B * Tm * m.d_model * es);
    r.tv = a.take<char>((size_t)tl * B * Tm * m.d_model * es);
    const int half = m.d_model / m.n_heads / 2;
    r.cosT = a.take<float>((size_t)c.max_pos * half);
    r.sinT = a.take<float>((size_t)c.max_pos * half);
    r.ropeT = a.take<float>((size_t)c.max_pos * 16 * 4 * 2);
    r.lp = a.take<float>((size_t)B * Tm * c.nitem);
    r.root = a.take<float>((size_t)B * c.nitem);
    if (keep) {
      c.reuse = true;
      c.lp_set[0] = r.lp;
      c.lp_set[1] = a.take<float>((size_t)B * Tm * c.nitem);
      c.prev_tpath = a.take<uint32_t>((size_t)B * Tm);
      c.prev_depth = a.take<int>((size_t)B * Tm);
      c.prev_n = a.take<int>(B);
      c.src = a.take<int>((size_t)B * Tm);
      c.fidx = a.take<int>((size_t)B * Tm);
      c.fcnt = a.take<int>(B);
    }
  }
  const size_t M = c.Mmax;
  c.x = a.take<float>(M * dmax);
  c.xn = a.take<char>(M * dmax * es);
  c.q = a.take<char>(M * dmax * es);
  c.ao = a.take<char>(M * dmax * es);
  c.h = a.take<char>(M * fmax * es);
  c.logits = a.take<float>(M * c.nitem);
  c.scratch = c.bf16 ? nullptr : a.take<float>(M * std::max(3 * dmax, 2 * fmax));
  c.part = c.bf16 ? a.take<float>(M * dmax) : nullptr;
  c.rows.M = a.take<int>(1);
  c.rows.user = a.take<int>(M);
  c.rows.token = a.take<int>(M);
  c.rows.pos = a.take<int>(M);
  c.rows.slot = a.take<int>(M);
  c.rows.nctx = a.take<int>(M);
  c.rows.anc = a.take<int>(M * 4);
  c.rows.nanc = a.take<int>(M);
  c.rows.user_off = a.take<int>(B + 1);
  const int K = cfg.K;
  c.state.t = a.take<int>(B);
  c.state.nb = a.take<int>(B);
  c.state.path = a.take<uint32_t>((size_t)B * K);
  c.state.trie = a.take<int>((size_t)B * K);
  c.state.score = a.take<float>((size_t)B * K);
  c.state.qscore = a.take<float>((size_t)B * K);
  c.state.beam_slot = a.take<int>((size_t)B * K);
  c.state.steps = a.take<int>(B);
  c.state.npath = a.take<int>(B);
  c.state.nfwd = a.take<int>(B);
  c.state.K = K;
  c.state.gamma = cfg.gamma;
  c.tree.max_nodes = Tm;
  c.tree.n_nodes = a.take<int>(B);
  c.tree.token = a.take<int>((size_t)B * Tm);
  c.tree.parent = a.take<int>((size_t)B * Tm);
  c.tree.depth = a.take<int>((size_t)B * Tm);
  c.tree.q_score = a.take<float>((size_t)B * Tm);
  c.tree.tpath = a.take<uint32_t>((size_t)B * Tm);
  c.tree.ttrie = a.take<int>((size_t)B * Tm);
  c.lo = a.take<int>(B);
  c.hi = a.take<int>(B);
  c.lvl_lo = a.take<int>(B);
  c.lvl_hi = a.take<int>(B);
  c.row_last = a.take<int>(B);
  c.Mb = a.take<int>(1);
  c.Mall = a.take<int>(1);
  c.plan_max = a.take<int>(1);
  c.err = a.take<int>(1);
  c.acc_tmp = a.take<int>(B);
  c.tafter_tmp = a.take<int>(B);
  c.keys = a.take<unsigned long long>((size_t)B * c.max_cand);
  const size_t nc = (size_t)B * c.max_cand;
  c.cand.path = a.take<uint32_t>(nc);
  c.cand.par = a.take<int>(nc);
  c.cand.cidx = a.take<int>(nc);
  c.cand.sp = a.take<float>(nc);
  c.cand.sq = a.take<float>(nc);
  c.relax.mode = cfg.mode;
  c.relax.tau = cfg.temperature;
  c.relax.k0 = (uint32_t)(cfg.seed & 0xFFFFFFFFu);
  c.relax.k1 = (uint32_t)(cfg.seed >> 32);
  c.relax.N = cfg.N;
  c.relax.zq = a.take<float>((size_t)B * (L + 1));
  c.relax.slot_node = a.take<int>((size_t)B * (L + 1) * K);
  c.relax.keys = c.keys;
  c.root_h = a.take<char>((size_t)B * std::max(cfg.draft.d_model, 1) * es);
  c.align_kslot = a.take<int>((size_t)B * L);
  c.loss_rows = a.take<float>(M);
}

atspeed_status bind_weights(ModelRt& r, const atspeed_weights* w, const char* who) {
  std::string s(who);
  if (!w || !w->tok_emb || !w->layers || !w->final_norm || !w->lm_head_item)
    return fail(ATSPEED_E_INVALID, s + " weights: null pointer");
  r.emb = w->tok_emb;
  r.final_norm = w->final_norm;
  r.lm_head = w->lm_head_item;
  r.layers.assign(w->layers, w->layers + (size_t)r.dims.n_layers * 9);
  for (const void* p : r.layers)
    if (!p) return fail(ATSPEED_E_INVALID, s + " weights: null layer pointer");
  r.present = true;
  return ATSPEED_OK;
}

atspeed_status upload_rope(atspeed_ctx& c, ModelRt& r) {
  const int dh = r.dh(), half = dh / 2;
  std::vector<float> cs((size_t)c.max_pos * half), sn((size_t)c.max_pos * half);
  for (int p = 0; p < c.max_pos; ++p)
    for (int i = 0; i < half; ++i) {
      double ang = (double)p * std::pow(10000.0, -2.0 * i / dh);
      cs[(size_t)p * half + i] = (float)std::cos(ang);
      sn[(size_t)p * half + i] = (float)std::sin(ang);
    }
  // the same values regrouped for the bf16 q/k/v epilogue: (cos, sin) of rotary
  // index 16*b + i at [pos][i][b], so a lane's four blocks are two 16-byte loads
  std::vector<float> rt((size_t)c.max_pos * 16 * 4 * 2, 0.f);
  for (int p = 0; p < c.max_pos; ++p)
    for (int i = 0; i < 16; ++i)
      for (int b = 0; b < 4; ++b) {
        const int ri = 16 * b + i;
        if (ri >= half) continue;
        rt[(((size_t)p * 16 + i) * 4 + b) * 2] = cs[(size_t)p * half + ri];
        rt[(((size_t)p * 16 + i) * 4 + b) * 2 + 1] = sn[(size_t)p * half + ri];
      }
  HIP_TRY(hipMemcpyAsync(r.cosT, cs.data(), cs.size() * 4, hipMemcpyHostToDevice, c.st));
  HIP_TRY(hipMemcpyAsync(r.sinT, sn.data(), sn.size() * 4, hipMemcpyHostToDevice, c.st));
  HIP_TRY(hipMemcpyAsync(r.ropeT, rt.data(), rt.size() * 4, hipMemcpyHostToDevice, c.st));
  HIP_TRY(hipStreamSynchronize(c.st));
  return ATSPEED_OK;
}

// One decoder forward over the planned rows.  prefill: K/V into the prefix cache,
// log-probs at each user's last position into r.root; else K/V into the tree
// buffer and log-probs into r.lp by tree slot (logits copied to dbg if given).
atspeed_status forward(atspeed_ctx& c, ModelRt& r, bool prefill, int Mmax, int Tq, float* dbg, int shared = 0) {
  const atspeed_model_dims& m = r.dims;
  const int d = m.d_model, f = m.d_ffn, H = m.n_heads, dh = r.dh();
  const int B = c.B;
  const size_t es = esize(c);
  hipStream_t st = c.st;
  // the marks below know which model they bracket (target launches forward
  // exactly Mmax rows, the draft's are sized by a bound)
  struct Current {
    atspeed_ctx& c;
    Current(atspeed_ctx& cc, const ModelRt& r) : c(cc) { c.fwd_model = &r; }
    ~Current() { c.fwd_model = nullptr; }
  } current(c, r);
  const double M = Mmax;
  // residual-stream capture (armed by atspeed_capture_hidden for one target
  // forward): the row plan now, x at every sublayer boundary below
  bool cap = c.cap_x != nullptr && &r == (c.cap_model == 1 ? &c.dft : &c.tgt);
  if (cap && c.cap_skip > 0) {
    --c.cap_skip;
    cap = false;
  }
  const int crow = cap ? std::min(Mmax, c.cap_rows) : 0;
  auto capture = [&](int idx) -> hipError_t {
    return hipMemcpyAsync(c.cap_x + (size_t)idx * c.cap_rows * d, c.x, (size_t)crow * d * sizeof(float),
                          hipMemcpyDeviceToDevice, st);
  };
  // bf16 activations: per layer [xn1 | q | k | v | ao | xn2] of [cap_rows][d], then a of [cap_rows][f];
  // after the layers the final norm's output [cap_rows][d]
  const bool cap_act = cap && c.cap_act != nullptr && c.bf16;
  const size_t act_layer = (size_t)c.cap_rows * (6 * (size_t)d + f);
  auto act = [&](int l, int part) -> bf16_t* { return c.cap_act + (size_t)l * act_layer + (size_t)part * c.cap_rows * d; };
  auto capture_act = [&](int l, int part, const void* src, int width) -> hipError_t {
    return hipMemcpyAsync(act(l, part), src, (size_t)crow * width * sizeof(bf16_t), hipMemcpyDeviceToDevice, st);
  };
  if (cap) {
    const int* src[3] = {c.rows.user, c.rows.pos, c.rows.slot};
    for (int i = 0; i < 3; ++i)
      HIP_TRY(hipMemcpyAsync(c.cap_plan + (size_t)i * c.cap_rows, src[i], (size_t)crow * sizeof(int),
                             hipMemcpyDeviceToDevice, st));
    HIP_TRY(hipMemcpyAsync(c.cap_plan + (size_t)3 * c.cap_rows, c.rows.M, sizeof(int), hipMemcpyDeviceToDevice, st));
  }
  MARK(ATSPEED_K_ROW);
  HIP_TRY(embed(c.bf16, r.emb, c.rows, Mmax, d, c.x, st));
  // bf16: the o and down projections split k at its midpoint (whole even
  // numbers of 64-column k-tiles), so 256x256 tiles fill the CUs at these
  // widths; the first half adds into x, the second goes to c.part, and the
  // next RMSNorm adds it and writes x back.  The split does not depend on the
  // row count, so neither does any row's arithmetic.
  float* part_o = c.bf16 && d % 256 == 0 ? c.part : nullptr;
  float* part_down = c.bf16 && f % 256 == 0 ? c.part : nullptr;
  for (int l = 0; l < m.n_layers; ++l) {
    const void* const* w = &r.layers[(size_t)l * 9];
    MARK(ATSPEED_K_ROW);
    HIP_TRY(rmsnorm(c.bf16, c.x, l > 0 ? part_down : nullptr, c.rows.M, Mmax, d, (const float*)w[0], c.xn, nullptr,
                    st));
    if (cap) HIP_TRY(capture(2 * l));       // the layer's input (the previous k-split half added)
    if (cap_act) HIP_TRY(capture_act(l, 0, c.xn, d));
    GemmCall g{};
    g.bf16 = c.bf16;
    g.Mmax = Mmax; g.Mdev = c.rows.M; g.scratch = c.scratch; g.rows = c.rows;
    g.cosT = r.cosT; g.sinT = r.sinT; g.ropeT = r.ropeT; g.d = d; g.dh = dh; g.H = H; g.Pmax = c.cfg.max_prefix;
    // q, k, v (+ rotary), k/v to their cache
    g.kind = GEMM_QKV; g.A = c.xn; g.lda = d; g.N = 3 * d; g.K = d;
    g.w0 = w[1]; g.w1 = w[2]; g.w2 = w[3]; g.split = d; g.q = c.q;
    char* pk = (char*)r.pk + (size_t)l * r.pkv_layer_stride * es;
    char* pv = (char*)r.pv + (size_t)l * r.pkv_layer_stride * es;
    char* tk = (char*)r.tk + (size_t)(r.kv_layer0 + l) * r.tkv_layer_stride * es;
    char* tv = (char*)r.tv + (size_t)(r.kv_layer0 + l) * r.tkv_layer_stride * es;
    g.kv_mode = prefill ? 0 : 1;
    g.kdst = prefill ? (void*)pk : (void*)tk;
    g.vdst = prefill ? (void*)pv : (void*)tv;
    MARK_F(ATSPEED_K_QKV, 2.0 * M * 3.0 * d * d);
    HIP_TRY(gemm(g, st));
    if (prefill && shared > 0 && B > 1) {  // users 1..B-1 take user 0's K/V of the shared positions
      launch_broadcast_prefix_kv(pk, pv, B, H, (size_t)c.cfg.max_prefix * dh * es, (size_t)shared * dh * es, st);
      HIP_TRY(hipGetLastError());
    }
    if (cap_act) {
      HIP_TRY(capture_act(l, 1, c.q, d));
      HIP_TRY(gather_kv_rows(prefill ? (void*)pk : (void*)tk, prefill ? (void*)pv : (void*)tv, c.rows, crow,
                             prefill ? 0 : 1, H, dh, c.cfg.max_prefix, act(l, 2), act(l, 3), st));
    }
    AttnCall at{};
    at.bf16 = c.bf16; at.q = c.q; at.pk = pk; at.pv = pv;
    at.tk = prefill ? nullptr : tk; at.tv = prefill ? nullptr : tv;
    at.out = c.ao; at.rows = c.rows; at.Mmax = Mmax; at.B = B; at.Tq = Tq;
    at.H = H; at.dh = dh; at.d = d; at.Pmax = c.cfg.max_prefix;
    MARK(ATSPEED_K_ATTN);
    HIP_TRY(attention(at, st));
    if (cap_act) HIP_TRY(capture_act(l, 4, c.ao, d));
    g.kind = GEMM_RESID; g.A = c.ao; g.lda = d; g.N = d; g.K = d; g.w0 = w[4]; g.out = c.x; g.ldo = d;
    g.part = part_o;
    MARK_F(ATSPEED_K_O, 2.0 * M * d * d);
    HIP_TRY(gemm(g, st));
    MARK(ATSPEED_K_ROW);
    HIP_TRY(rmsnorm(c.bf16, c.x, part_o, c.rows.M, Mmax, d, (const float*)w[5], c.xn, nullptr, st));
    if (cap) HIP_TRY(capture(2 * l + 1));   // after the attention sublayer
    if (cap_act) HIP_TRY(capture_act(l, 5, c.xn, d));
    g.kind = GEMM_GU; g.A = c.xn; g.lda = d; g.N = 2 * f; g.K = d; g.w0 = w[6]; g.w1 = w[7]; g.split = f; g.hout = c.h;
    MARK_F(ATSPEED_K_GU, 2.0 * M * 2.0 * f * d);
    HIP_TRY(gemm(g, st));
    if (cap_act) HIP_TRY(capture_act(l, 6, c.h, f));
    g.kind = GEMM_RESID; g.A = c.h; g.lda = f; g.N = d; g.K = f; g.w0 = w[8]; g.out = c.x; g.ldo = d;
    g.part = part_down;
    MARK_F(ATSPEED_K_DOWN, 2.0 * M * f * d);
    HIP_TRY(gemm(g, st));
  }
  // final norm + item rows of the output head + log-softmax
  const int* Mfin = prefill ? c.Mb : c.rows.M;
  const int Mmf = prefill ? B : Mmax;
  MARK(ATSPEED_K_ROW);
  HIP_TRY(rmsnorm(c.bf16, c.x, part_down, Mfin, Mmf, d, r.final_norm, c.xn, prefill ? c.row_last : nullptr, st));
  // after the last layer (a prefill writes no whole residual back: its final
  // norm runs on each user's last row only)
  if (cap && !prefill) HIP_TRY(capture(2 * m.n_layers));
  if (cap_act && !prefill) HIP_TRY(capture_act(m.n_layers, 0, c.xn, d));
  if (cap) { c.cap_x = nullptr; c.cap_act = nullptr; c.cap_plan = nullptr; c.cap_rows = 0; }
  GemmCall g{};
  g.kind = GEMM_STORE; g.bf16 = c.bf16; g.A = c.xn; g.lda = d; g.Mmax = Mmf; g.Mdev = Mfin;
  g.N = c.nitem; g.K = d; g.w0 = r.lm_head; g.out = c.logits; g.ldo = c.nitem; g.scratch = c.scratch;
  MARK_F(ATSPEED_K_LMHEAD, 2.0 * Mmf * c.nitem * d);
  HIP_TRY(gemm(g, st));
  MARK(ATSPEED_K_ROW);
  if (prefill) HIP_TRY(log_softmax_rows(c.logits, c.Mb, B, c.nitem, nullptr, r.root, dbg, st));
  else HIP_TRY(log_softmax_rows(c.logits, c.rows.M, Mmax, c.nitem, c.rows.slot, r.lp, dbg, st));
  MARK(-1);
  // the draft's root hidden states, for recomputing its root log-probs when its
  // item head is trained (atspeed_align_step)
  if (prefill && &r == &c.dft) HIP_TRY(hipMemcpyAsync(c.root_h, c.xn, (size_t)B * d * es, hipMemcpyDeviceToDevice, st));
  return ATSPEED_OK;
}

atspeed_status read_err(atspeed_ctx& c, int* out) {
  HIP_TRY(hipMemcpyAsync(out, c.err, sizeof(int), hipMemcpyDeviceToHost, c.st));
  HIP_TRY(hipStreamSynchronize(c.st));
  return ATSPEED_OK;
}

// carry: the decode loop's own verify, which may take the nodes the previous
// verify of the loop forwarded (with tree-KV reuse configured).
atspeed_status tree_forward(atspeed_ctx& c, float* dbg_logits, bool carry = false) {
  HIP_TRY(hipMemsetAsync(c.err, 0, sizeof(int), c.st));
  HIP_TRY(hipMemsetAsync(c.lo, 0, sizeof(int) * c.B, c.st));
  MARK(ATSPEED_K_SELECT);
  launch_tree_index(c.tree, c.trie, c.state, c.B, c.cfg.target.item_base, c.cfg.codebook, c.cfg.L, c.err, c.st);
  HIP_TRY(hipGetLastError());
  const bool use_prev = c.reuse && carry && c.carry_ok;
  const int nset = c.kv_cur ^ 1;   // this verify's buffer set
  if (c.reuse) {
    c.carry_ok = false;            // until this verify has completed
    launch_carry_match(c.tree, c.state, c.prev_tpath, c.prev_depth, use_prev ? c.prev_n : nullptr, c.src, c.fidx,
                       c.fcnt, c.B, c.st);
    HIP_TRY(hipGetLastError());
    launch_plan_tree(c.tree, c.lo, c.fcnt, c.B, c.P, c.rows, c.plan_max, c.st, c.fidx);
  } else {
    launch_plan_tree(c.tree, c.lo, c.state.nfwd, c.B, c.P, c.rows, c.plan_max, c.st);
  }
  HIP_TRY(hipGetLastError());
  // One read-back per forward: the validity word, the row count and the largest
  // per-user row count, so a malformed tree never reaches the forward and every
  // launch of the forward is sized to the rows it has.
  int info[3] = {0, 0, 0};
  HIP_TRY(hipMemcpyAsync(&info[0], c.err, sizeof(int), hipMemcpyDeviceToHost, c.st));
  HIP_TRY(hipMemcpyAsync(&info[1], c.rows.M, sizeof(int), hipMemcpyDeviceToHost, c.st));
  HIP_TRY(hipMemcpyAsync(&info[2], c.plan_max, sizeof(int), hipMemcpyDeviceToHost, c.st));
  HIP_TRY(hipStreamSynchronize(c.st));
  if (info[0]) return fail(ATSPEED_E_INVALID, "malformed tree (code " + std::to_string(info[0]) + ")");
  if (c.reuse) {
    ModelRt& r = c.tgt;
    const int nl = r.dims.n_layers;
    const size_t es = esize(c), layer_bytes = r.tkv_layer_stride * es;
    r.kv_layer0 = nset * nl;
    r.lp = c.lp_set[nset];
    if (use_prev) {
      launch_carry_copy(c.src, c.state.nfwd, c.B, c.Tmax, nl, layer_bytes, r.dims.d_model * (int)es,
                        (char*)r.tk + (size_t)c.kv_cur * nl * layer_bytes,
                        (char*)r.tv + (size_t)c.kv_cur * nl * layer_bytes, (char*)r.tk + (size_t)nset * nl * layer_bytes,
                        (char*)r.tv + (size_t)nset * nl * layer_bytes, c.lp_set[c.kv_cur], c.lp_set[nset], c.nitem,
                        c.st);
      HIP_TRY(hipGetLastError());
    }
  }
  if (info[1] > 0) ST_TRY(forward(c, c.tgt, false, info[1], info[2], dbg_logits));
  c.rows_fwd += info[1];
  if (c.reuse) {
    // this tree's forwarded and carried nodes are slots [0, nfwd) of the new set
    const size_t n = (size_t)c.B * c.Tmax;
    HIP_TRY(hipMemcpyAsync(c.prev_tpath, c.tree.tpath, n * 4, hipMemcpyDeviceToDevice, c.st));
    HIP_TRY(hipMemcpyAsync(c.prev_depth, c.tree.depth, n * 4, hipMemcpyDeviceToDevice, c.st));
    HIP_TRY(hipMemcpyAsync(c.prev_n, c.state.nfwd, (size_t)c.B * 4, hipMemcpyDeviceToDevice, c.st));
    c.kv_cur = nset;
    c.carry_ok = carry;
  }
  return ATSPEED_OK;
}

}  // namespace

// ---------------------------------------------------------------- allocation-free accept
// Scratch of atspeed_accept_noalloc: one copy per GPU, held until the process
// ends.  In host code the name only stands for the symbol; its device address is
// taken once per device with hipGetSymbolAddress and used everywhere instead.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
std::mutex g_scratch_mu;
constexpr int kMaxDevices = 64;
unsigned char* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of the static scratch (taken on first use).
atspeed_status static_scratch_address(unsigned char** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(ATSPEED_E_DEVICE, "device index out of range for the static scratch");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    g_scratch_ptr[dev] = static_cast<unsigned char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return ATSPEED_OK;
}
}  // namespace

// ====================================================================== ABI

extern "C" {

const char* atspeed_last_error(void) { return g_err.c_str(); }

atspeed_status atspeed_workspace_bytes(const atspeed_config* cfg, const atspeed_catalog* cat, size_t* bytes) {
  if (!bytes) return fail(ATSPEED_E_INVALID, "bytes is null");
  ST_TRY(check_config(cfg));
  HostTrie t;
  ST_TRY(build_trie(*cfg, cat, t));
  atspeed_ctx c;
  Arena a{nullptr};
  layout(c, *cfg, (int)t.code.size(), a);
  *bytes = a.off + 256;
  return ATSPEED_OK;
}

atspeed_status atspeed_create(const atspeed_config* cfg, const atspeed_weights* target, const atspeed_weights* draft,
                              const atspeed_catalog* cat, void* ws, size_t ws_bytes, atspeed_ctx** out) {
  if (!out) return fail(ATSPEED_E_INVALID, "out is null");
  *out = nullptr;
  ST_TRY(check_config(cfg));
  if (!ws) return fail(ATSPEED_E_WORKSPACE, "workspace is null");
  if (reinterpret_cast<uintptr_t>(ws) & 255) return fail(ATSPEED_E_WORKSPACE, "workspace is not 256-byte aligned");
  HostTrie t;
  ST_TRY(build_trie(*cfg, cat, t));
  size_t need = 0;
  {
    atspeed_ctx tmp;
    Arena a{nullptr};
    layout(tmp, *cfg, (int)t.code.size(), a);
    need = a.off + 256;
  }
  if (ws_bytes < need) return fail(ATSPEED_E_WORKSPACE, "workspace too small: need " + std::to_string(need) + " bytes");
  atspeed_ctx* c = new atspeed_ctx();
  c->cfg = *cfg;
  c->st = (hipStream_t)cfg->stream;
  Arena a{(char*)ws};
  layout(*c, *cfg, (int)t.code.size(), a);
  c->htrie = std::move(t);
  atspeed_status s = bind_weights(c->tgt, target, "target");
  if (s == ATSPEED_OK && draft && cfg->draft.n_layers > 0) s = bind_weights(c->dft, draft, "draft");
  auto bail = [&](atspeed_status e) { delete c; return e; };
  if (s != ATSPEED_OK) return bail(s);
  const size_t nn = c->htrie.code.size();
  hipError_t e = hipMemcpyAsync((void*)c->trie.code, c->htrie.code.data(), nn * 4, hipMemcpyHostToDevice, c->st);
  if (e == hipSuccess) e = hipMemcpyAsync((void*)c->trie.first, c->htrie.first.data(), nn * 4, hipMemcpyHostToDevice, c->st);
  if (e == hipSuccess) e = hipMemcpyAsync((void*)c->trie.cnt, c->htrie.cnt.data(), nn * 4, hipMemcpyHostToDevice, c->st);
  if (e == hipSuccess) e = hipMemsetAsync(c->state.t, 0, sizeof(int) * cfg->max_batch, c->st);
  if (e == hipSuccess) e = hipMemsetAsync(c->state.steps, 0, sizeof(int) * cfg->max_batch, c->st);
  if (e == hipSuccess) e = hipMemsetAsync(c->tree.n_nodes, 0, sizeof(int) * cfg->max_batch, c->st);
  if (e == hipSuccess) e = hipStreamSynchronize(c->st);
  if (e != hipSuccess) return bail(fail(ATSPEED_E_DEVICE, std::string("create: ") + hipGetErrorString(e)));
  s = upload_rope(*c, c->tgt);
  if (s == ATSPEED_OK && c->dft.present) s = upload_rope(*c, c->dft);
  if (s == ATSPEED_OK) s = static_scratch_address(&c->static_scratch);
  if (s != ATSPEED_OK) return bail(s);
  *out = c;
  return ATSPEED_OK;
}

void atspeed_destroy(atspeed_ctx* ctx) { delete ctx; }



static atspeed_status prefill_impl(atspeed_ctx* c, int32_t B, int32_t P, const int32_t* prefix, float* root_logits,
                                   bool with_draft) {
  if (!c) return fail(ATSPEED_E_INVALID, "ctx is null");
  if (!prefix) return fail(ATSPEED_E_INVALID, "prefix is null");
  if (B < 1 || B > c->cfg.max_batch) return fail(ATSPEED_E_SHAPE, "B out of range");
  if (P < 1 || P > c->cfg.max_prefix) return fail(ATSPEED_E_SHAPE, "P out of range");
  c->B = B;
  c->P = P;
  // Positions every user shares with user 0 (a common prompt) are forwarded
  // once: user 0 computes them, the others copy its K/V.  Their hidden states
  // depend only on those tokens, and a row's results do not depend on its batch,
  // so the caches and logits are the same as with every row forwarded.  Each
  // user keeps at least its last position (its root logits).
  int S = 0;
  if (B > 1) {
    launch_common_prefix(prefix, B, P, c->plan_max, c->st);
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipMemcpyAsync(&S, c->plan_max, sizeof(int), hipMemcpyDeviceToHost, c->st));
    HIP_TRY(hipStreamSynchronize(c->st));
    S = std::min(S, P - 1);
  }
  const int M = P + (B - 1) * (P - S);
  std::vector<int> last(B), sizes{B, B * c->Tmax};
  for (int u = 0; u < B; ++u) last[u] = u == 0 ? P - 1 : P + u * (P - S) - 1;
  HIP_TRY(hipMemcpyAsync(c->row_last, last.data(), B * 4, hipMemcpyHostToDevice, c->st));
  HIP_TRY(hipMemcpyAsync(c->Mb, &sizes[0], 4, hipMemcpyHostToDevice, c->st));
  HIP_TRY(hipMemcpyAsync(c->Mall, &sizes[1], 4, hipMemcpyHostToDevice, c->st));
  launch_plan_prefix(prefix, B, P, S, c->rows, c->st);
  HIP_TRY(hipGetLastError());
  c->dft_prefilled = false;
  ST_TRY(forward(*c, c->tgt, true, M, P, root_logits, S));
  if (with_draft && c->dft.present) ST_TRY(forward(*c, c->dft, true, M, P, nullptr, S));
  c->shared_prefix = S;
  HIP_TRY(hipMemsetAsync(c->state.t, 0, sizeof(int) * B, c->st));
  HIP_TRY(hipMemsetAsync(c->state.steps, 0, sizeof(int) * B, c->st));
  std::vector<int> ones(B, 1);
  HIP_TRY(hipMemcpyAsync(c->state.nb, ones.data(), B * 4, hipMemcpyHostToDevice, c->st));
  HIP_TRY(hipMemsetAsync(c->tree.n_nodes, 0, sizeof(int) * B, c->st));
  HIP_TRY(hipStreamSynchronize(c->st));  // host vectors above go out of scope
  c->prefilled = true;
  c->dft_prefilled = with_draft && c->dft.present;
  c->drafted = false;
  c->carry_ok = false;
  c->align_ready = false;
  return ATSPEED_OK;
}

atspeed_status atspeed_prefill(atspeed_ctx* c, int32_t B, int32_t P, const int32_t* prefix, float* root_logits) {
  return prefill_impl(c, B, P, prefix, root_logits, true);
}

atspeed_status atspeed_draft(atspeed_ctx* c) {
  if (!c) return fail(ATSPEED_E_INVALID, "ctx is null");
  if (!c->dft.present) return fail(ATSPEED_E_STATE, "context has no draft model");
  if (!c->prefilled) return fail(ATSPEED_E_STATE, "draft before prefill");
  if (!c->dft_prefilled) return fail(ATSPEED_E_STATE, "draft after a target-only prefill (atspeed_target_search)");
  const atspeed_config& cf = c->cfg;
  const int B = c->B, L = cf.L;
  launch_tree_from_beams(c->state, c->tree, c->trie, B, cf.target.item_base, cf.codebook, L, c->st);
  HIP_TRY(hipGetLastError());
  // draft log-probs along the Y_t paths (none at t = 0), then the beams' draft scores
  HIP_TRY(hipMemsetAsync(c->lo, 0, sizeof(int) * B, c->st));
  launch_plan_tree(c->tree, c->lo, c->state.npath, B, c->P, c->rows, nullptr, c->st);
  HIP_TRY(hipGetLastError());
  // Row bounds of the draft forwards (the row counts themselves stay on the
  // device): the Y_t paths are prefixes of at most K beams at depths 1..t < L,
  // and a drafted level holds at most N nodes per user (the strict and the
  // paper's relaxed draft keep at most N; the exact relaxed draft keeps the
  // distinct winners of K draws, and N >= K).  The bounds size the launches and
  // choose the GEMM tiles, so they are kept tight.
  c->align_ready = false;  // the tree is rebuilt below
  const int path_rows = std::max(1, cf.K * (L - 1)), level_rows = std::max(1, cf.N);
  ST_TRY(forward(*c, c->dft, false, B * path_rows, path_rows, nullptr));
  launch_draft_beam_scores(c->state, c->tree, c->dft.lp, c->dft.root, c->nitem, cf.codebook, L, B, c->st);
  HIP_TRY(hipGetLastError());
  for (int j = 1; j <= std::min(cf.gamma, L); ++j) {
    if (cf.mode == ATSPEED_STRICT)
      launch_draft_select(c->state, c->tree, c->trie, c->dft.lp, c->dft.root, c->nitem, cf.target.item_base,
                          cf.codebook, L, j, cf.N, c->lvl_lo, c->lvl_hi, c->keys, c->max_cand, B, c->st);
    else
      launch_draft_relaxed(c->state, c->tree, c->trie, c->dft.lp, c->dft.root, c->nitem, cf.target.item_base,
                           cf.codebook, L, j, c->lvl_lo, c->lvl_hi, c->cand, c->max_cand, c->relax, B, c->st);
    HIP_TRY(hipGetLastError());
    if (j < std::min(cf.gamma, L)) {  // log-probs of the new level feed the next one
      launch_plan_tree(c->tree, c->lvl_lo, c->lvl_hi, B, c->P, c->rows, nullptr, c->st);
      HIP_TRY(hipGetLastError());
      ST_TRY(forward(*c, c->dft, false, B * level_rows, level_rows, nullptr));
    }
  }
  c->drafted = true;
  return ATSPEED_OK;
}

atspeed_status atspeed_get_tree(atspeed_ctx* c, atspeed_tree* out) {
  if (!c || !out) return fail(ATSPEED_E_INVALID, "null argument");
  out->max_nodes = c->tree.max_nodes;
  out->n_nodes = c->tree.n_nodes;
  out->token = c->tree.token;
  out->parent = c->tree.parent;
  out->depth = c->tree.depth;
  out->q_score = c->tree.q_score;
  return ATSPEED_OK;
}

atspeed_status atspeed_tree_logits(atspeed_ctx* c, float* logits) {
  if (!c || !logits) return fail(ATSPEED_E_INVALID, "null argument");
  if (!c->prefilled) return fail(ATSPEED_E_STATE, "tree_logits before prefill");
  ST_TRY(tree_forward(*c, logits));
  HIP_TRY(hipStreamSynchronize(c->st));
  return ATSPEED_OK;
}

static atspeed_status accept_on(atspeed_ctx* c, const float* lpt, const float* roott, int32_t* accepted,
                                int32_t* t_after) {
  const atspeed_config& cf = c->cfg;
  HIP_TRY(mark(*c, ATSPEED_K_SELECT));
  if (cf.mode == ATSPEED_STRICT) {
    launch_verify_strict(c->state, c->tree, c->trie, lpt, roott, c->nitem, cf.codebook, cf.L, c->keys, c->max_cand,
                         accepted ? accepted : c->acc_tmp, t_after ? t_after : c->tafter_tmp, c->B, c->st);
  } else {
    if (!c->drafted) return fail(ATSPEED_E_STATE, "relaxed verification needs the context's own draft of this step");
    launch_verify_relaxed(c->state, c->tree, c->trie, lpt, roott, c->dft.lp, c->dft.root, c->nitem, cf.codebook, cf.L,
                          c->cand, c->max_cand, c->relax, accepted ? accepted : c->acc_tmp,
                          t_after ? t_after : c->tafter_tmp, c->B, c->st);
  }
  HIP_TRY(hipGetLastError());
  HIP_TRY(mark(*c, -1));
  return ATSPEED_OK;
}

static atspeed_status verify_step(atspeed_ctx* c, int32_t* accepted, int32_t* t_after, float* logits, bool carry) {
  if (!c) return fail(ATSPEED_E_INVALID, "ctx is null");
  if (!c->prefilled) return fail(ATSPEED_E_STATE, "verify before prefill");
  ST_TRY(tree_forward(*c, logits, carry));
  ST_TRY(accept_on(c, c->tgt.lp, c->tgt.root, accepted, t_after));
  c->drafted = false;
  return ATSPEED_OK;
}

atspeed_status atspeed_verify(atspeed_ctx* c, int32_t* accepted, int32_t* t_after, float* logits) {
  return verify_step(c, accepted, t_after, logits, false);
}

atspeed_status atspeed_accept(atspeed_ctx* c, const float* logits, const float* root_logits, int32_t* accepted,
                              int32_t* t_after) {
  if (!c || !logits || !root_logits) return fail(ATSPEED_E_INVALID, "null argument");
  if (!c->prefilled) return fail(ATSPEED_E_STATE, "accept before prefill");
  HIP_TRY(hipMemsetAsync(c->err, 0, sizeof(int), c->st));
  launch_tree_index(c->tree, c->trie, c->state, c->B, c->cfg.target.item_base, c->cfg.codebook, c->cfg.L, c->err, c->st);
  HIP_TRY(hipGetLastError());
  int err = 0;
  ST_TRY(read_err(*c, &err));
  if (err) return fail(ATSPEED_E_INVALID, "malformed tree (code " + std::to_string(err) + ")");
  // log-softmax of the caller's logits into the slot-indexed buffers (row = slot)
  HIP_TRY(log_softmax_rows(logits, c->Mall, c->B * c->Tmax, c->nitem, nullptr, c->tgt.lp, nullptr, c->st));
  HIP_TRY(log_softmax_rows(root_logits, c->Mb, c->B, c->nitem, nullptr, c->tgt.root, nullptr, c->st));
  ST_TRY(accept_on(c, c->tgt.lp, c->tgt.root, accepted, t_after));
  HIP_TRY(hipStreamSynchronize(c->st));
  return ATSPEED_OK;
}

atspeed_status atspeed_accept_noalloc(atspeed_ctx* c, const float* logits, const float* root_logits,
                                      int32_t* accepted, int32_t* t_after) {
  if (!c || !logits || !root_logits) return fail(ATSPEED_E_INVALID, "null argument");
  if (!c->prefilled) return fail(ATSPEED_E_STATE, "accept before prefill");
  const atspeed_config& cf = c->cfg;
  const bool relaxed = cf.mode != ATSPEED_STRICT;
  if (relaxed && !c->drafted) return fail(ATSPEED_E_STATE, "relaxed verification needs the context's own draft of this step");
  if (!c->static_scratch) return fail(ATSPEED_E_DEVICE, "static scratch address unknown");
  // carve the static scratch: error word, log-prob rows by slot, root rows,
  // selection keys, relaxed candidate buffers
  const size_t B = c->B, rows = B * c->Tmax, nc = B * c->max_cand;
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off = (off + bytes + 255) & ~size_t(255); return o; };
  const size_t o_err = take(sizeof(int)), o_lp = take(rows * c->nitem * 4), o_root = take(B * c->nitem * 4);
  const size_t o_keys = take(nc * 8);
  size_t o_cand[5] = {0, 0, 0, 0, 0};
  if (relaxed)
    for (size_t& o : o_cand) o = take(nc * 4);
  if (off > kStaticScratchBytes)
    return fail(ATSPEED_E_WORKSPACE, "accept_noalloc needs " + std::to_string(off) + " bytes of scratch for this batch; " +
                                         "the static scratch holds " + std::to_string(kStaticScratchBytes));
  unsigned char* base = c->static_scratch;
  int* err = reinterpret_cast<int*>(base + o_err);
  float* lp = reinterpret_cast<float*>(base + o_lp);
  float* root = reinterpret_cast<float*>(base + o_root);
  unsigned long long* keys = reinterpret_cast<unsigned long long*>(base + o_keys);
  HIP_TRY(hipMemsetAsync(err, 0, sizeof(int), c->st));
  launch_tree_index(c->tree, c->trie, c->state, c->B, cf.target.item_base, cf.codebook, cf.L, err, c->st);
  HIP_TRY(hipGetLastError());
  int bad = 0;
  HIP_TRY(hipMemcpyAsync(&bad, err, sizeof(int), hipMemcpyDeviceToHost, c->st));
  HIP_TRY(hipStreamSynchronize(c->st));
  if (bad) return fail(ATSPEED_E_INVALID, "malformed tree (code " + std::to_string(bad) + ")");
  HIP_TRY(log_softmax_rows(logits, c->Mall, c->B * c->Tmax, c->nitem, nullptr, lp, nullptr, c->st));
  HIP_TRY(log_softmax_rows(root_logits, c->Mb, c->B, c->nitem, nullptr, root, nullptr, c->st));
  int* acc = accepted ? accepted : c->acc_tmp;
  int* ta = t_after ? t_after : c->tafter_tmp;
  if (!relaxed) {
    launch_verify_strict(c->state, c->tree, c->trie, lp, root, c->nitem, cf.codebook, cf.L, keys, c->max_cand, acc,
                         ta, c->B, c->st);
  } else {
    RelaxArgs ra = c->relax;
    ra.keys = keys;
    CandBuf cb{reinterpret_cast<uint32_t*>(base + o_cand[0]), reinterpret_cast<int*>(base + o_cand[1]),
               reinterpret_cast<int*>(base + o_cand[2]), reinterpret_cast<float*>(base + o_cand[3]),
               reinterpret_cast<float*>(base + o_cand[4])};
    launch_verify_relaxed(c->state, c->tree, c->trie, lp, root, c->dft.lp, c->dft.root, c->nitem, cf.codebook, cf.L,
                          cb, c->max_cand, ra, acc, ta, c->B, c->st);
  }
  HIP_TRY(hipGetLastError());
  HIP_TRY(hipStreamSynchronize(c->st));
  return ATSPEED_OK;
}

atspeed_status atspeed_logprobs(atspeed_ctx* c, int32_t model, float* lp, float* root) {
  if (!c || !lp || !root) return fail(ATSPEED_E_INVALID, "null argument");
  if (model != 0 && model != 1) return fail(ATSPEED_E_INVALID, "model must be 0 (target) or 1 (draft)");
  if (!c->prefilled) return fail(ATSPEED_E_STATE, "logprobs before prefill");
  const ModelRt& m = model == 0 ? c->tgt : c->dft;
  if (!m.present) return fail(ATSPEED_E_STATE, "context has no draft model");
  if (model == 1 && !c->dft_prefilled) return fail(ATSPEED_E_STATE, "the last prefill did not run the draft");
  const size_t row = (size_t)c->nitem * sizeof(float);
  HIP_TRY(hipMemcpyAsync(lp, m.lp, (size_t)c->B * c->Tmax * row, hipMemcpyDeviceToDevice, c->st));
  HIP_TRY(hipMemcpyAsync(root, m.root, (size_t)c->B * row, hipMemcpyDeviceToDevice, c->st));
  HIP_TRY(hipStreamSynchronize(c->st));
  return ATSPEED_OK;
}

atspeed_status atspeed_get_state(atspeed_ctx* c, int32_t B, int32_t* t, int32_t* nbeams, int32_t* paths, float* scores) {
  if (!c || !t || !nbeams || !paths || !scores) return fail(ATSPEED_E_INVALID, "null argument");
  if (B < 1 || B > c->cfg.max_batch) return fail(ATSPEED_E_SHAPE, "B out of range");
  const int K = c->cfg.K, L = c->cfg.L;
  std::vector<uint32_t> pk((size_t)B * K);
  HIP_TRY(hipMemcpyAsync(t, c->state.t, B * 4, hipMemcpyDeviceToHost, c->st));
  HIP_TRY(hipMemcpyAsync(nbeams, c->state.nb, B * 4, hipMemcpyDeviceToHost, c->st));
  HIP_TRY(hipMemcpyAsync(pk.data(), c->state.path, pk.size() * 4, hipMemcpyDeviceToHost, c->st));
  HIP_TRY(hipMemcpyAsync(scores, c->state.score, (size_t)B * K * 4, hipMemcpyDeviceToHost, c->st));
  HIP_TRY(hipStreamSynchronize(c->st));
  for (size_t i = 0; i < pk.size(); ++i)
    for (int l = 0; l < L; ++l) paths[i * L + l] = (pk[i] >> (8 * (3 - l))) & 0xFF;
  return ATSPEED_OK;
}

atspeed_status atspeed_set_state(atspeed_ctx* c, int32_t B, const int32_t* t, const int32_t* nbeams,
                                 const int32_t* paths, const float* scores) {
  if (!c || !t || !nbeams || !paths || !scores) return fail(ATSPEED_E_INVALID, "null argument");
  if (B < 1 || B != c->B) return fail(ATSPEED_E_SHAPE, "B must equal the prefilled batch");
  const int K = c->cfg.K, L = c->cfg.L;
  std::vector<uint32_t> pk((size_t)B * K, 0);
  std::vector<int> tr((size_t)B * K, 0);
  for (int u = 0; u < B; ++u) {
    if (t[u] < 0 || t[u] > L) return fail(ATSPEED_E_INVALID, "t out of range");
    if (nbeams[u] < 1 || nbeams[u] > K) return fail(ATSPEED_E_INVALID, "nbeams out of range");
    if (t[u] == 0 && nbeams[u] != 1) return fail(ATSPEED_E_INVALID, "t = 0 holds one (empty) beam");
    for (int k = 0; k < nbeams[u]; ++k) {
      int node = 0;
      uint32_t p = 0;
      for (int l = 0; l < t[u]; ++l) {
        int code = paths[((size_t)u * K + k) * L + l];
        if (code < 0 || code >= c->cfg.codebook) return fail(ATSPEED_E_INVALID, "path code out of range");
        node = c->htrie.child(node, code);
        if (node < 0) return fail(ATSPEED_E_INVALID, "beam is not a catalog prefix");
        p |= (uint32_t)code << (8 * (3 - l));
      }
      pk[(size_t)u * K + k] = p;
      tr[(size_t)u * K + k] = node;
    }
  }
  HIP_TRY(hipMemcpyAsync(c->state.t, t, B * 4, hipMemcpyHostToDevice, c->st));
  HIP_TRY(hipMemcpyAsync(c->state.nb, nbeams, B * 4, hipMemcpyHostToDevice, c->st));
  HIP_TRY(hipMemcpyAsync(c->state.path, pk.data(), pk.size() * 4, hipMemcpyHostToDevice, c->st));
  HIP_TRY(hipMemcpyAsync(c->state.trie, tr.data(), tr.size() * 4, hipMemcpyHostToDevice, c->st));
  HIP_TRY(hipMemcpyAsync(c->state.score, scores, (size_t)B * K * 4, hipMemcpyHostToDevice, c->st));
  HIP_TRY(hipStreamSynchronize(c->st));
  return ATSPEED_OK;
}

// The users' final beams as lists: items [B, K, L] codes, scores [B, K], counts [B] (device).
static atspeed_status write_lists(atspeed_ctx* c, int32_t B, int32_t* items, float* scores, int32_t* n_items) {
  launch_write_lists(c->state, B, c->cfg.K, c->cfg.L, items, scores, n_items, c->st);
  HIP_TRY(hipGetLastError());
  HIP_TRY(hipStreamSynchronize(c->st));
  return ATSPEED_OK;
}

atspeed_status atspeed_decode_topk(atspeed_ctx* c, int32_t B, int32_t P, const int32_t* prefix, int32_t* items,
                                   float* scores, int32_t* n_items, atspeed_stats* stats) {
  if (!c) return fail(ATSPEED_E_INVALID, "ctx is null");
  if (!items || !scores || !n_items) return fail(ATSPEED_E_INVALID, "null output");
  if (!c->dft.present) return fail(ATSPEED_E_STATE, "context has no draft model");
  hipEvent_t ev[2];
  const bool timing = stats != nullptr;
  if (timing) {
    HIP_TRY(hipEventCreate(&ev[0]));
    HIP_TRY(hipEventCreate(&ev[1]));
    stats->n_steps = 0;
    stats->rows_target = 0;
    stats->ms_prefill = stats->ms_draft = stats->ms_verify = 0;
    HIP_TRY(hipEventRecord(ev[0], c->st));
  }
  auto lap = [&](double* acc) -> atspeed_status {
    if (!timing) return ATSPEED_OK;
    HIP_TRY(hipEventRecord(ev[1], c->st));
    HIP_TRY(hipEventSynchronize(ev[1]));
    float ms = 0;
    HIP_TRY(hipEventElapsedTime(&ms, ev[0], ev[1]));
    *acc += ms;
    HIP_TRY(hipEventRecord(ev[0], c->st));
    return ATSPEED_OK;
  };
  ST_TRY(atspeed_prefill(c, B, P, prefix, nullptr));
  ST_TRY(lap(timing ? &stats->ms_prefill : nullptr));
  c->rows_fwd = 0;
  const int L = c->cfg.L;
  std::vector<int> acc(B), ta(B);
  for (int step = 0; step < L; ++step) {
    if (step == 0 && c->cfg.sd_start_level == 1) {
      // level 1 from the prefill: a verify over a tree with no nodes selects the
      // target's level from the root log-probs (the bonus level of zero accepted)
      HIP_TRY(hipMemsetAsync(c->tree.n_nodes, 0, sizeof(int) * B, c->st));
    } else {
      ST_TRY(atspeed_draft(c));
      ST_TRY(lap(timing ? &stats->ms_draft : nullptr));
    }
    ST_TRY(verify_step(c, c->acc_tmp, c->tafter_tmp, nullptr, true));
    HIP_TRY(hipMemcpyAsync(acc.data(), c->acc_tmp, B * 4, hipMemcpyDeviceToHost, c->st));
    HIP_TRY(hipMemcpyAsync(ta.data(), c->tafter_tmp, B * 4, hipMemcpyDeviceToHost, c->st));
    HIP_TRY(hipStreamSynchronize(c->st));
    ST_TRY(lap(timing ? &stats->ms_verify : nullptr));
    if (timing) {
      if (stats->accepted) std::copy(acc.begin(), acc.end(), stats->accepted + (size_t)step * c->cfg.max_batch);
      if (stats->t_after) std::copy(ta.begin(), ta.end(), stats->t_after + (size_t)step * c->cfg.max_batch);
      stats->n_steps = step + 1;
      stats->rows_target = c->rows_fwd;
    }
    if (std::all_of(ta.begin(), ta.end(), [&](int v) { return v >= L; })) break;
  }
  if (timing) {
    hipEventDestroy(ev[0]);
    hipEventDestroy(ev[1]);
  }
  return write_lists(c, B, items, scores, n_items);
}

atspeed_status atspeed_target_search(atspeed_ctx* c, int32_t B, int32_t P, const int32_t* prefix, int32_t* items,
                                     float* scores, int32_t* n_items, int32_t* step_items, int32_t* step_lens,
                                     int32_t* step_n) {
  if (!c) return fail(ATSPEED_E_INVALID, "ctx is null");
  if (!items || !scores || !n_items) return fail(ATSPEED_E_INVALID, "null output");
  if ((step_items != nullptr) != (step_lens != nullptr) || (step_items != nullptr) != (step_n != nullptr))
    return fail(ATSPEED_E_INVALID, "step_items, step_lens and step_n are given together or not at all");
  ST_TRY(prefill_impl(c, B, P, prefix, nullptr, false));
  const atspeed_config& cf = c->cfg;
  const int L = cf.L;
  if (step_n) HIP_TRY(hipMemsetAsync(step_n, 0, sizeof(int) * B, c->st));
  for (int l = 0; l < L; ++l) {
    // the tree of the Y_t paths alone: the verify has no drafted level, so it
    // takes the target's TopK of level t + 1 (at t = 0 from the prefill's root)
    launch_tree_from_beams(c->state, c->tree, c->trie, B, cf.target.item_base, cf.codebook, L, c->st);
    HIP_TRY(hipGetLastError());
    ST_TRY(tree_forward(*c, nullptr, true));
    launch_verify_strict(c->state, c->tree, c->trie, c->tgt.lp, c->tgt.root, c->nitem, cf.codebook, L, c->keys,
                         c->max_cand, c->acc_tmp, c->tafter_tmp, B, c->st);
    HIP_TRY(hipGetLastError());
    if (step_items) {
      launch_append_beams(c->state, B, L, step_items, step_lens, step_n, c->st);
      HIP_TRY(hipGetLastError());
    }
  }
  return write_lists(c, B, items, scores, n_items);
}

atspeed_status atspeed_align_data(atspeed_ctx* c, int32_t S, const int32_t* items, const int32_t* lens,
                                  const int32_t* n_items, const atspeed_align_args* a) {
  if (!c || !items || !n_items || !a) return fail(ATSPEED_E_INVALID, "null argument");
  if (!a->ctx_weight || !a->label_weight || !a->root_weight || !a->log_pK || !a->lp_target || !a->root_target)
    return fail(ATSPEED_E_INVALID, "align_data: null batch buffer");
  if (S < 1) return fail(ATSPEED_E_SHAPE, "align_data: S must be positive");
  if (!c->prefilled || !c->dft_prefilled) return fail(ATSPEED_E_STATE, "align_data needs atspeed_prefill first");
  if (!c->dft.present) return fail(ATSPEED_E_STATE, "context has no draft model");
  const atspeed_config& cf = c->cfg;
  const int B = c->B, L = cf.L;
  c->align_ready = false;
  c->drafted = false;
  // every user back at t = 0 with the empty beam (the tree carries no beams)
  std::vector<int> ones(B, 1);
  HIP_TRY(hipMemsetAsync(c->state.t, 0, sizeof(int) * B, c->st));
  HIP_TRY(hipMemcpyAsync(c->state.nb, ones.data(), B * 4, hipMemcpyHostToDevice, c->st));
  HIP_TRY(hipMemsetAsync(c->err, 0, sizeof(int), c->st));
  launch_align_tree(items, lens, n_items, S, c->tree, c->trie, B, L, cf.target.item_base, cf.codebook, a->ctx_weight,
                    a->label_weight, a->root_weight, c->align_kslot, c->err, c->st);
  HIP_TRY(hipGetLastError());
  int err = 0;
  ST_TRY(read_err(*c, &err));   // synchronises: the host vector above is consumed
  if (err)
    return fail(ATSPEED_E_INVALID, "align_data: a count outside 1..S, a length outside 1..L, a last sequence "
                                   "shorter than L, a prefix outside the catalog, or more prefixes than max_nodes");
  // the target over every context (validated again by the tree walk of the forward)
  ST_TRY(tree_forward(*c, nullptr));
  const size_t row = (size_t)c->nitem * sizeof(float);
  HIP_TRY(hipMemcpyAsync(a->lp_target, c->tgt.lp, (size_t)B * c->Tmax * row, hipMemcpyDeviceToDevice, c->st));
  HIP_TRY(hipMemcpyAsync(a->root_target, c->tgt.root, (size_t)B * row, hipMemcpyDeviceToDevice, c->st));
  launch_align_logpk(items, n_items, c->align_kslot, a->lp_target, a->root_target, B, S, L, cf.codebook, c->nitem,
                     a->log_pK, c->st);
  HIP_TRY(hipGetLastError());
  HIP_TRY(hipStreamSynchronize(c->st));
  c->align_ready = true;
  return ATSPEED_OK;
}

atspeed_status atspeed_align_step(atspeed_ctx* c, const atspeed_align_args* a, double* loss) {
  if (!c || !a) return fail(ATSPEED_E_INVALID, "null argument");
  if (!a->ctx_weight || !a->label_weight || !a->root_weight || !a->log_pK || !a->lp_target || !a->root_target ||
      !a->master || !a->adam_m || !a->adam_v || !a->grad)
    return fail(ATSPEED_E_INVALID, "align_step: null buffer");
  if (a->mode != 0 && a->mode != 1) return fail(ATSPEED_E_INVALID, "align_step: mode must be 0 (S) or 1 (R)");
  if (!(a->alpha >= 0.f && a->alpha <= 1.f)) return fail(ATSPEED_E_INVALID, "align_step: alpha outside [0, 1]");
  if (a->step < 1) return fail(ATSPEED_E_INVALID, "align_step: step counts from 1");
  if (!(a->lr >= 0.f) || !(a->beta1 >= 0.f && a->beta1 < 1.f) || !(a->beta2 >= 0.f && a->beta2 < 1.f) ||
      !(a->eps > 0.f) || !(a->weight_decay >= 0.f))
    return fail(ATSPEED_E_INVALID, "align_step: optimizer hyper-parameter out of range");
  if (!c->align_ready) return fail(ATSPEED_E_STATE, "align_step needs atspeed_align_data after the last prefill or draft");
  const atspeed_config& cf = c->cfg;
  ModelRt& r = c->dft;
  const int B = c->B, L = cf.L, d = r.dims.d_model;
  // the draft's root log-probs with the current head
  {
    GemmCall g{};
    g.kind = GEMM_STORE; g.bf16 = c->bf16; g.A = c->root_h; g.lda = d; g.Mmax = B; g.Mdev = c->Mb;
    g.N = c->nitem; g.K = d; g.w0 = r.lm_head; g.out = c->logits; g.ldo = c->nitem; g.scratch = c->scratch;
    HIP_TRY(gemm(g, c->st));
    HIP_TRY(log_softmax_rows(c->logits, c->Mb, B, c->nitem, nullptr, r.root, nullptr, c->st));
  }
  // the context rows: every tree node of depth < L (the leaves of depth L are
  // labels only)
  HIP_TRY(hipMemsetAsync(c->err, 0, sizeof(int), c->st));
  HIP_TRY(hipMemsetAsync(c->lo, 0, sizeof(int) * B, c->st));
  launch_tree_index(c->tree, c->trie, c->state, B, cf.target.item_base, cf.codebook, L, c->err, c->st);
  HIP_TRY(hipGetLastError());
  launch_plan_tree(c->tree, c->lo, c->state.nfwd, B, c->P, c->rows, c->plan_max, c->st);
  HIP_TRY(hipGetLastError());
  int info[3] = {0, 0, 0};
  HIP_TRY(hipMemcpyAsync(&info[0], c->err, sizeof(int), hipMemcpyDeviceToHost, c->st));
  HIP_TRY(hipMemcpyAsync(&info[1], c->rows.M, sizeof(int), hipMemcpyDeviceToHost, c->st));
  HIP_TRY(hipMemcpyAsync(&info[2], c->plan_max, sizeof(int), hipMemcpyDeviceToHost, c->st));
  HIP_TRY(hipStreamSynchronize(c->st));
  if (info[0]) return fail(ATSPEED_E_INVALID, "align_step: the context tree is malformed (code " + std::to_string(info[0]) + ")");
  const int M = info[1];
  if (B + M > c->Mmax) return fail(ATSPEED_E_SHAPE, "align_step: more context rows than the forward holds");
  if (M > 0) ST_TRY(forward(*c, r, false, M, info[2], nullptr));   // hidden rows in c->xn, log-probs by slot
  AlignRows ar{c->rows.M, c->rows.user, c->rows.slot, r.lp, r.root, a->lp_target, a->root_target, a->ctx_weight,
               a->label_weight, a->root_weight, a->log_pK};
  launch_align_grad(ar, c->trie, c->tree, B, M, c->nitem, cf.codebook, L, cf.K, a->mode, a->alpha, c->logits,
                    c->loss_rows, c->st);
  HIP_TRY(hipGetLastError());
  launch_head_grad(c->bf16, c->logits, c->root_h, c->xn, c->rows.M, B, c->nitem, d, a->grad, c->st);
  HIP_TRY(hipGetLastError());
  if (a->hidden_out) {
    launch_align_hidden(c->bf16, c->root_h, c->xn, c->rows.slot, c->rows.M, B, M, d, a->hidden_out, c->st);
    HIP_TRY(hipGetLastError());
  }
  launch_adamw(c->bf16, a->master, a->adam_m, a->adam_v, a->grad, const_cast<void*>(r.lm_head), (size_t)c->nitem * d,
               a->lr, a->beta1, a->beta2, a->eps, a->weight_decay, a->step, c->st);
  HIP_TRY(hipGetLastError());
  std::vector<float> lr((size_t)B + M);
  HIP_TRY(hipMemcpyAsync(lr.data(), c->loss_rows, lr.size() * 4, hipMemcpyDeviceToHost, c->st));
  HIP_TRY(hipStreamSynchronize(c->st));
  if (loss) {
    double sum = 0.0;
    for (float v : lr) sum += v;
    *loss = sum;
  }
  return ATSPEED_OK;
}

atspeed_status atspeed_mixed_search(atspeed_ctx* c, float lambda, int32_t B, int32_t P, const int32_t* prefix,
                                    int32_t* items, float* scores, int32_t* n_items, int32_t* step_items,
                                    int32_t* step_lens, int32_t* step_n) {
  if (!c) return fail(ATSPEED_E_INVALID, "ctx is null");
  if (!items || !scores || !n_items) return fail(ATSPEED_E_INVALID, "null output");
  if (!(lambda >= 0.f && lambda <= 1.f)) return fail(ATSPEED_E_INVALID, "mixed_search: lambda outside [0, 1]");
  if ((step_items != nullptr) != (step_lens != nullptr) || (step_items != nullptr) != (step_n != nullptr))
    return fail(ATSPEED_E_INVALID, "step_items, step_lens and step_n are given together or not at all");
  if (!c->dft.present) return fail(ATSPEED_E_STATE, "context has no draft model");
  ST_TRY(prefill_impl(c, B, P, prefix, nullptr, true));
  const atspeed_config& cf = c->cfg;
  const int L = cf.L, path_rows = std::max(1, cf.K * (L - 1));
  if (step_n) HIP_TRY(hipMemsetAsync(step_n, 0, sizeof(int) * B, c->st));
  for (int l = 0; l < L; ++l) {
    // the Y_t paths alone, through the target and the draft
    launch_tree_from_beams(c->state, c->tree, c->trie, B, cf.target.item_base, cf.codebook, L, c->st);
    HIP_TRY(hipGetLastError());
    ST_TRY(tree_forward(*c, nullptr, true));
    HIP_TRY(hipMemsetAsync(c->lo, 0, sizeof(int) * B, c->st));
    launch_plan_tree(c->tree, c->lo, c->state.npath, B, c->P, c->rows, nullptr, c->st);
    HIP_TRY(hipGetLastError());
    ST_TRY(forward(*c, c->dft, false, B * path_rows, path_rows, nullptr));
    // the mixture into the draft's rows, then the strict TopK of the next level
    if (l == 0) launch_mix_logprobs(c->dft.root, c->tgt.root, nullptr, B, 1, c->nitem, lambda, c->st);
    else launch_mix_logprobs(c->dft.lp, c->tgt.lp, c->state.npath, B, c->Tmax, c->nitem, lambda, c->st);
    HIP_TRY(hipGetLastError());
    launch_verify_strict(c->state, c->tree, c->trie, c->dft.lp, c->dft.root, c->nitem, cf.codebook, L, c->keys,
                         c->max_cand, c->acc_tmp, c->tafter_tmp, B, c->st);
    HIP_TRY(hipGetLastError());
    if (step_items) {
      launch_append_beams(c->state, B, L, step_items, step_lens, step_n, c->st);
      HIP_TRY(hipGetLastError());
    }
  }
  c->dft_prefilled = false;   // the draft's root row now holds the mixture
  c->drafted = false;
  return write_lists(c, B, items, scores, n_items);
}

atspeed_status atspeed_capture_hidden(atspeed_ctx* c, int32_t model, int32_t skip, float* x, void* act,
                                      int32_t* plan, int32_t max_rows) {
  if (!c) return fail(ATSPEED_E_INVALID, "null context");
  if (model != 0 && model != 1) return fail(ATSPEED_E_INVALID, "capture_hidden: model is 0 (target) or 1 (draft)");
  if (skip < 0) return fail(ATSPEED_E_INVALID, "capture_hidden: skip < 0");
  if (model == 1 && !c->dft.present) return fail(ATSPEED_E_STATE, "capture_hidden: context has no draft model");
  if (x == nullptr && act == nullptr && plan == nullptr) {
    c->cap_x = nullptr; c->cap_act = nullptr; c->cap_plan = nullptr; c->cap_rows = 0;
    return ATSPEED_OK;
  }
  if (!x || !plan || max_rows <= 0)
    return fail(ATSPEED_E_INVALID, "capture_hidden: x and plan buffers and max_rows > 0 needed");
  if (act && !c->bf16) return fail(ATSPEED_E_INVALID, "capture_hidden: activations are captured for bf16 models only");
  c->cap_x = x; c->cap_act = (bf16_t*)act; c->cap_plan = plan; c->cap_rows = max_rows; c->cap_model = model;
  c->cap_skip = skip;
  return ATSPEED_OK;
}

atspeed_status atspeed_set_timing(atspeed_ctx* c, int32_t enable) {
  if (!c) return fail(ATSPEED_E_INVALID, "ctx is null");
  HIP_TRY(fold_timing(*c));
  c->timing_mask = (uint32_t)enable & ATSPEED_TIME_ALL;
  c->timing_target_only = (enable & ATSPEED_TIME_TARGET_ONLY) != 0;
  for (int k = 0; k < ATSPEED_K_COUNT; ++k) { c->t_ms[k] = 0; c->t_n[k] = 0; c->t_flop[k] = 0; }
  return ATSPEED_OK;
}

atspeed_status atspeed_get_timing(atspeed_ctx* c, atspeed_kernel_times* out) {
  if (!c || !out) return fail(ATSPEED_E_INVALID, "null argument");
  HIP_TRY(fold_timing(*c));
  for (int k = 0; k < ATSPEED_K_COUNT; ++k) {
    out->ms[k] = c->t_ms[k];
    out->launches[k] = c->t_n[k];
    out->gflop[k] = c->t_flop[k] * 1e-9;
  }
  return ATSPEED_OK;
}

}  // extern "C"
