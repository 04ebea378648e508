// Host engine behind the C ABI of include/ee.h: argument validation, the
// paged KV allocator, per-sequence state, host<->device staging and the
// launch sequence of one verification step.

#include <hip/hip_runtime.h>

#include <math.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>
#include <new>
#include <string>
#include <vector>

#include "../../include/ee.h"
#include "kernels.h"

namespace {

constexpr int PAGE = 64;
constexpr int SPLIT = 256;
constexpr int MAX_K = 512;        // longest linear draft
constexpr int MAX_TREE = 64;      // largest draft tree (one node per lane of a wave)
constexpr size_t ALIGN = 256;

size_t up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

// Scratch of ee_verify_noalloc: the step's attention split states and GEMM
// slice partials, in a static device array (one per GPU the library runs on,
// held until the process ends) instead of the caller's workspace.
constexpr size_t NOALLOC_SCRATCH_BYTES = size_t(16) << 20;
constexpr int MAX_DEVICES = 64;

thread_local std::string g_err = "no error";

}  // namespace

static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

namespace {

std::mutex g_scratch_mu;
void* g_scratch_addr[MAX_DEVICES] = {};   // device address of `scratch` on each GPU

// The device address of this GPU's `scratch` (the array's name is only a
// host-side stand-in), looked up once per device with that device current.
hipError_t scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return hipSuccess;
}

struct Seq {
  bool live = false;
  int len = 0;
  int pending = -1;
  std::vector<int> pages;   // page of positions [64 i, 64 i + 64)
};

// Byte offsets of every buffer inside the three caller allocations.
struct Layout {
  int Tmax, Rmax, MT, G, max_splits, pages_per_seq, ptable_len, n_pages;
  // packed arena
  size_t embed, lm_head, final_gain, layers0, per_layer, l_wqkv, l_wo, l_wgu, l_wd, l_again, l_fgain,
      packed_total;
  // workspace
  size_t h, ssq, xbuf, x2buf, ssqt, zbuf, q, part, gpart, logits, amax, greedy, verdict, rowstat, ebuf, result, stage, rope, ws_total;
  // staging sub-offsets (relative to `stage`)
  size_t s_tok, s_pos, s_prow, s_slot, s_path, s_ptable, s_info, s_eps, s_unif, s_sparam, stage_bytes;
  size_t kv_layer, kv_total;
};

bool valid_cfg(const ee_model_config* c, std::string* why) {
  auto bad = [&](const char* m) { if (why) *why = m; return false; };
  if (!c) return bad("config is NULL");
  if (c->dtype != EE_F32 && c->dtype != EE_BF16) return bad("dtype must be EE_F32 or EE_BF16");
  if (c->n_layers < 1 || c->d_model < 1 || c->n_heads < 1 || c->n_kv_heads < 1 || c->ffn < 1 ||
      c->vocab < 1)
    return bad("every model dimension must be positive");
  if (c->head_dim != 64 && c->head_dim != 128) return bad("head_dim must be 64 or 128");
  if (c->dtype == EE_F32 && c->head_dim != 64) return bad("fp32 models need head_dim 64");
  if (c->n_heads % c->n_kv_heads) return bad("n_heads must be a multiple of n_kv_heads");
  const int ks = c->dtype == EE_BF16 ? 32 : 16;
  if (c->d_model > 8192 || c->ffn > 32768 || (int64_t)c->n_heads * c->head_dim > 32768)   // (no int overflow)
    return bad("d_model <= 8192, ffn and n_heads*head_dim <= 32768");
  if (c->d_model % ks || c->ffn % ks || (c->n_heads * c->head_dim) % ks || c->vocab % ks)
    return bad("d_model, ffn, n_heads*head_dim and vocab must be multiples of 32 (bf16) / 16 (f32)");
  if (c->page_size != PAGE) return bad("page_size must be 64");
  if (c->k_max < 0 || c->k_max > MAX_K) return bad("k_max must be in [0, 512]");
  if (c->max_ctx < 1 || c->max_seqs < 1) return bad("max_ctx and max_seqs must be positive");
  if (c->max_ctx > 8192) return bad("max_ctx must be at most 8192");
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f)) return bad("rms_eps >= 0 and rope_theta > 0");
  if ((c->n_heads / c->n_kv_heads) * (c->k_max + 1) > 64 * 16 * 16)
    return bad("too many query columns per KV head");
  {
    // one layer of the KV pool is addressed with 32-bit buffer offsets
    const size_t pages = (size_t)((c->max_ctx + PAGE - 1) / PAGE) * c->max_seqs;
    const size_t layer = pages * 2 * c->n_kv_heads * PAGE * c->head_dim * (c->dtype == EE_BF16 ? 2 : 4);
    if (layer >= (size_t(1) << 31)) return bad("one layer of the KV pool must stay below 2 GiB");
  }
  {
    // the packed LM head and embedding are addressed with 32-bit buffer offsets
    const size_t head = (size_t)c->vocab * c->d_model * (c->dtype == EE_BF16 ? 2 : 4);
    if (head >= (size_t(1) << 31)) return bad("vocab * d_model of the LM head must stay below 2 GiB");
  }
  {
    // GEMM slice partials of one block are written through 32-bit buffer offsets
    const int dt = c->dtype == EE_BF16 ? ee::DT_BF16 : ee::DT_F32;
    const size_t rows = (size_t)(c->k_max + 1) * c->max_seqs;
    const size_t n_max = std::max({(size_t)c->vocab, (size_t)2 * c->ffn,
                                   (size_t)(c->n_heads + 2 * c->n_kv_heads) * c->head_dim});
    const size_t sk = (size_t)std::max(ee::gemm_slices_for(c->d_model, dt), ee::gemm_slices_for(c->ffn, dt));
    if (sk * rows * n_max * 4 >= (size_t(1) << 31))
      return bad("the GEMM partials of one block must stay below 2 GiB (fewer sequences or draft tokens)");
  }
  return true;
}

// Columns of the largest GEMM slice-partial array of a row: max over the
// projections of K slices x output features.
size_t partial_cols(const ee_model_config& g) {
  const int dt = g.dtype == EE_BF16 ? ee::DT_BF16 : ee::DT_F32;
  const size_t d = g.d_model, qd = (size_t)g.n_heads * g.head_dim, F = g.ffn;
  const size_t qkvN = qd + 2 * (size_t)g.n_kv_heads * g.head_dim;
  size_t mx = 0;
  mx = std::max(mx, (size_t)ee::gemm_slices_for((int)d, dt) * qkvN);
  mx = std::max(mx, (size_t)ee::gemm_slices_for((int)qd, dt) * d);
  mx = std::max(mx, (size_t)ee::gemm_slices_for((int)d, dt) * 2 * F);
  mx = std::max(mx, (size_t)ee::gemm_slices_for((int)F, dt) * d);
  mx = std::max(mx, (size_t)ee::gemm_slices_for((int)d, dt) * (size_t)g.vocab);
  return mx;
}

Layout make_layout(const ee_model_config* c) {
  Layout L{};
  const size_t esz = c->dtype == EE_BF16 ? 2 : 4;
  const int ks = c->dtype == EE_BF16 ? 32 : 16;
  const size_t d = c->d_model, hd = c->head_dim, H = c->n_heads, Hkv = c->n_kv_heads;
  const size_t F = c->ffn, V = c->vocab;
  L.Tmax = c->k_max + 1;
  L.Rmax = L.Tmax * c->max_seqs;   // a block holds up to max_seqs sequences
  L.MT = (L.Rmax + 15) / 16;
  L.G = c->n_heads / c->n_kv_heads;
  L.max_splits = (c->max_ctx + SPLIT - 1) / SPLIT + 1;
  L.pages_per_seq = (c->max_ctx + PAGE - 1) / PAGE;
  L.ptable_len = (L.pages_per_seq + 3) & ~3;   // 16-byte loads of page numbers
  L.n_pages = L.pages_per_seq * c->max_seqs;
  // packed arena
  size_t o = 0;
  L.embed = o; o += up(V * d * esz);
  L.lm_head = o; o += up(V * d * esz);
  L.final_gain = o; o += up(d * 4);
  L.layers0 = o;
  L.l_wqkv = 0;
  size_t lo = 0;
  lo += up((H + 2 * Hkv) * hd * d * esz); L.l_wo = lo;
  lo += up(d * H * hd * esz); L.l_wgu = lo;
  lo += up(2 * F * d * esz); L.l_wd = lo;
  lo += up(d * F * esz); L.l_again = lo;
  lo += up(d * 4); L.l_fgain = lo;
  lo += up(d * 4);
  L.per_layer = lo;
  L.packed_total = o + lo * c->n_layers;
  // workspace
  const size_t Tpad = (size_t)L.MT * 16;
  const size_t xcols = std::max(d, H * hd);
  o = 0;
  L.h = o; o += up(L.Rmax * d * 4);
  L.ssq = o; o += up((size_t)L.Rmax * 8 * 4);
  L.xbuf = o; o += up(Tpad * xcols * esz);
  L.x2buf = o; o += up(Tpad * d * esz);
  L.ssqt = o; o += up((size_t)L.Rmax * (d / 16) * 4);
  L.zbuf = o; o += up(Tpad * F * esz);
  L.q = o; o += up(L.Rmax * H * hd * esz);
  L.part = o; o += up((size_t)L.max_splits * Hkv * L.Rmax * L.G * (hd + 2) * 4);
  // split-K partials of the largest GEMM: [slices][Rmax][N]
  L.gpart = o; o += up(partial_cols(*c) * L.Rmax * 4);
  L.logits = o; o += up(L.Rmax * V * 4);
  L.amax = o; o += up(L.Rmax * ((V + 2047) / 2048) * 8 * 8);
  L.greedy = o; o += up(L.Rmax * 4);
  L.verdict = o; o += up(L.Rmax * 4);
  L.rowstat = o; o += up((size_t)L.Rmax * 2 * 8);
  L.ebuf = o; o += up((size_t)L.Rmax * V * 8);
  L.result = o; o += up((size_t)c->max_seqs * (2 + c->k_max) * 4);
  // staging block: read from its pinned host mirror by the block's first kernel
  size_t so = 0;
  L.s_tok = so; so += L.Rmax * 4;
  L.s_pos = so; so += L.Rmax * 4;
  L.s_prow = so; so += L.Rmax * 4;
  L.s_slot = so; so += L.Rmax * 4;
  L.s_path = so; so += L.Rmax * 64;
  so = (so + 15) & ~(size_t)15;   // 16-byte loads of page numbers
  L.s_ptable = so; so += (size_t)c->max_seqs * L.ptable_len * 4;
  L.s_info = so; so += (size_t)c->max_seqs * 4 * 4;
  L.s_eps = so; so += (size_t)L.Rmax * 4;
  L.s_unif = so; so += (size_t)L.Rmax * 4;
  so = (so + 15) & ~(size_t)15;
  L.s_sparam = so; so += 16;
  L.stage_bytes = up(so);
  L.stage = o; o += L.stage_bytes;
  L.rope = o; o += up((size_t)c->max_ctx * (hd / 2) * 8);
  L.ws_total = o;
  (void)ks;
  // KV pool: [layer][page][2][Hkv][64 * hd]
  L.kv_layer = (size_t)L.n_pages * 2 * Hkv * PAGE * hd * esz;
  L.kv_total = L.kv_layer * c->n_layers;
  return L;
}

}  // namespace

struct ee_ctx {
  ee_model_config cfg;
  Layout lay;
  hipStream_t user_st = nullptr;     // caller's stream (ee_create work)
  hipStream_t st = nullptr;          // library stream of every later call
  hipEvent_t ev_user = nullptr;      // orders `st` after the caller's stream
  struct Captured {
    hipGraphExec_t exec;
    int prof_pairs;                  // event pairs recorded by the graph's own nodes
  };
  // (T, B, mode, attention splits, profiling mask)
  std::map<std::tuple<int, int, int, int, uint32_t>, Captured> graphs;
  bool graphs_ok = true;             // capture works on this stream
  bool graphs_on = true;             // ee_use_graphs
  unsigned char* packed = nullptr;
  unsigned char* pool = nullptr;
  unsigned char* ws = nullptr;
  std::vector<ee::LayerPtrs> layers;
  ee::Model m{};
  ee::Work w{};
  std::vector<Seq> seqs;
  std::vector<int> free_pages;
  unsigned char* h_stage = nullptr;   // pinned mirror of the staging block
  int* h_result = nullptr;            // pinned
  uint32_t* d_stage_src = nullptr;    // device-visible addresses of h_stage and h_result
  int* d_result_dst = nullptr;
  int last_T = 0;
  int dev = -1;                       // GPU of the context (current at ee_create)
  unsigned char* scratch = nullptr;   // that GPU's static scratch array (ee_verify_noalloc)
  unsigned char* cap = nullptr;       // ee_capture buffer (test aid) and its size
  size_t cap_bytes = 0;
  std::string err = "no error";
  // profiling
  ee::Prof prof;
  std::vector<hipEvent_t> events;
  std::vector<int> ev_cls;
  double prof_ms[ee::PC_N] = {};
  int64_t prof_n[ee::PC_N] = {};
};

namespace {

int fail(ee_ctx* c, int code, const std::string& msg) {
  if (c) c->err = msg; else g_err = msg;
  return code;
}

int hip_fail(ee_ctx* c, hipError_t e, const char* where) {
  return fail(c, EE_EHIP, std::string(where) + ": " + hipGetErrorString(e));
}

#define HIP_TRY(ctx, expr)                                      \
  do {                                                          \
    hipError_t e_ = (expr);                                     \
    if (e_ != hipSuccess) return hip_fail((ctx), e_, #expr);    \
  } while (0)

void bind_work(ee_ctx* c) {
  const Layout& L = c->lay;
  unsigned char* ws = c->ws;
  ee::Work& w = c->w;
  w.h = reinterpret_cast<float*>(ws + L.h);
  w.ssq = reinterpret_cast<float*>(ws + L.ssq);
  w.xbuf = reinterpret_cast<uint4*>(ws + L.xbuf);
  w.x2buf = reinterpret_cast<uint4*>(ws + L.x2buf);
  w.ssqt = reinterpret_cast<float*>(ws + L.ssqt);
  w.zbuf = reinterpret_cast<uint4*>(ws + L.zbuf);
  w.q = ws + L.q;
  w.attn_part = reinterpret_cast<float*>(ws + L.part);
  w.part = reinterpret_cast<float*>(ws + L.gpart);
  w.logits = reinterpret_cast<float*>(ws + L.logits);
  w.amax = reinterpret_cast<unsigned long long*>(ws + L.amax);
  w.greedy = reinterpret_cast<int*>(ws + L.greedy);
  w.verdict = reinterpret_cast<int*>(ws + L.verdict);
  w.rowstat = reinterpret_cast<double*>(ws + L.rowstat);
  w.ebuf = reinterpret_cast<double*>(ws + L.ebuf);
  w.result = reinterpret_cast<int*>(ws + L.result);
  unsigned char* sb = ws + L.stage;
  w.path = sb + L.s_path;
  w.tok = reinterpret_cast<int*>(sb + L.s_tok);
  w.pos = reinterpret_cast<int*>(sb + L.s_pos);
  w.prow = reinterpret_cast<int*>(sb + L.s_prow);
  w.slot = reinterpret_cast<int*>(sb + L.s_slot);
  w.ptable = reinterpret_cast<int*>(sb + L.s_ptable);
  w.info = reinterpret_cast<int*>(sb + L.s_info);
  w.eps = reinterpret_cast<float*>(sb + L.s_eps);
  w.unif = reinterpret_cast<float*>(sb + L.s_unif);
  w.sparam = sb + L.s_sparam;
  w.ptable_len = L.ptable_len;
  w.rec = 2 + c->cfg.k_max;
  w.max_splits = L.max_splits;
}

// Give `s` pages for positions [0, upto); returns false (and takes nothing)
// when the pool runs dry.
bool reserve_pages(ee_ctx* c, Seq& s, int upto, int* added) {
  const int need = (upto + PAGE - 1) / PAGE;
  const int have = (int)s.pages.size();
  *added = 0;
  if (need <= have) return true;
  if ((int)c->free_pages.size() < need - have) return false;
  for (int i = have; i < need; ++i) {
    s.pages.push_back(c->free_pages.back());
    c->free_pages.pop_back();
  }
  *added = need - have;
  return true;
}

void unreserve(ee_ctx* c, Seq& s, int n) {
  for (int i = 0; i < n; ++i) {
    c->free_pages.push_back(s.pages.back());
    s.pages.pop_back();
  }
}

int check_seq(ee_ctx* c, int seq) {
  if (!c) return fail(nullptr, EE_EINVAL, "context is NULL");
  if (seq < 0 || seq >= c->cfg.max_seqs) return fail(c, EE_EINVAL, "sequence index out of range");
  return EE_OK;
}

// The staging words a block of this shape reads: the rows' tokens, positions,
// parents and slots, the trees' paths, the sequences' page tables and step
// state, and the draws and parameters of stochastic verification.
ee::StageCopy stage_ranges(const ee_ctx* c, const ee::Step& step) {
  const Layout& L = c->lay;
  ee::StageCopy sc{};
  sc.src = c->d_stage_src;
  sc.dst = reinterpret_cast<uint32_t*>(c->ws + L.stage);
  const size_t R = (size_t)step.B * step.T;
  auto add = [&](size_t off, size_t words) {
    sc.off[sc.n] = (int)(off / 4);
    sc.len[sc.n] = (int)words;
    sc.total += (int)words;
    ++sc.n;
  };
  add(L.s_tok, R);
  add(L.s_pos, R);
  add(L.s_prow, R);
  add(L.s_slot, R);
  if (step.mode == 2) add(L.s_path, R * 16);
  add(L.s_ptable, (size_t)step.B * L.ptable_len);
  add(L.s_info, (size_t)step.B * 4);
  if (step.mode == 4) {
    add(L.s_eps, R);
    add(L.s_unif, R);
    add(L.s_sparam, 4);
  }
  return sc;
}

// The kernels of one block, in launch order: staging in, forward, acceptance
// (+ tree compaction), results out.
hipError_t launch_block(ee_ctx* c, const ee::Step& step, ee::Prof* prof, const ee::Work& w) {
  hipError_t e;
  if ((e = ee::run_stage_in(stage_ranges(c, step), c->st)) != hipSuccess) return e;
  if ((e = ee::run_forward(c->m, w, step, prof, c->st)) != hipSuccess) return e;
  if ((e = ee::run_accept(c->m, w, step, prof, c->st)) != hipSuccess) return e;
  if (step.mode == 2 && (e = ee::run_compact(c->m, w, step, prof, c->st)) != hipSuccess) return e;
  return ee::run_result_out(w, step.B, c->d_result_dst, c->st);
}

constexpr size_t MAX_GRAPHS = 512;   // captured block shapes kept at once

// Captured graph of a (T, B, mode, splits) block shape, built on first use
// (profiling events, when enabled, become event-record nodes of the graph);
// nullptr if capture is unavailable (the block then runs eagerly).  The
// attention grid is sized to the block's splits, so a context that grows
// past a multiple of 256 positions captures the shape again; past MAX_GRAPHS
// shapes the cache starts over (every call waits for its graph, so none is
// in flight).
const ee_ctx::Captured* block_graph(ee_ctx* c, const ee::Step& step, ee::Prof* prof) {
  if (!c->graphs_ok || !c->graphs_on) return nullptr;
  const auto key = std::make_tuple(step.T, step.B, step.mode, step.splits, prof ? prof->mask : 0u);
  auto it = c->graphs.find(key);
  if (it != c->graphs.end()) return &it->second;
  if (c->graphs.size() >= MAX_GRAPHS) {
    for (auto& kv : c->graphs) (void)hipGraphExecDestroy(kv.second.exec);
    c->graphs.clear();
  }
  hipGraph_t g = nullptr;
  hipGraphExec_t ge = nullptr;
  if (hipStreamBeginCapture(c->st, hipStreamCaptureModeThreadLocal) != hipSuccess) {
    c->graphs_ok = false;
    return nullptr;
  }
  if (prof) prof->used = 0;
  const hipError_t le = launch_block(c, step, prof, c->w);
  const hipError_t ce = hipStreamEndCapture(c->st, &g);
  if (le != hipSuccess || ce != hipSuccess || !g || hipGraphInstantiate(&ge, g, nullptr, nullptr, 0) != hipSuccess) {
    if (g) (void)hipGraphDestroy(g);
    (void)hipGetLastError();
    c->graphs_ok = false;
    return nullptr;
  }
  (void)hipGraphDestroy(g);
  auto& slot = c->graphs[key];
  slot.exec = ge;
  slot.prof_pairs = prof ? prof->used : 0;
  return &slot;
}

// Order the context's stream after the work enqueued on the caller's stream.
// An idle caller stream (the usual case) needs no event, whose record and wait
// cost ~15 us of host time per call.
int order_after_user(ee_ctx* c) {
  const hipError_t q = hipStreamQuery(c->user_st);
  if (q == hipSuccess) return EE_OK;
  if (q != hipErrorNotReady) return hip_fail(c, q, "hipStreamQuery");
  HIP_TRY(c, hipEventRecord(c->ev_user, c->user_st));
  HIP_TRY(c, hipStreamWaitEvent(c->st, c->ev_user, 0));
  return EE_OK;
}

// Stage the per-sequence state (page tables, committed lengths, the KV slot
// of every row) in the pinned mirror, run the block of B sequences of T rows
// whose tokens, positions and parents the caller staged (its kernels read the
// mirror and write the results to h_result, record b at h_result + b *
// (2 + k_max)) and wait for it.  Mode 3 uses the top-k size and dynamic flag
// given for every sequence.
// `scratch_work`: buffers of the block when they are not the context's own
// (ee_verify_noalloc); such a block runs without graph replay.
int run_block(ee_ctx* c, Seq* const* seqs, int B, int T, int mode, int top_k = 0, int dynamic = 0,
              const ee::Work* scratch_work = nullptr) {
  const Layout& L = c->lay;
  int* ptab = reinterpret_cast<int*>(c->h_stage + L.s_ptable);
  int* info = reinterpret_cast<int*>(c->h_stage + L.s_info);
  int* slot = reinterpret_cast<int*>(c->h_stage + L.s_slot);
  int splits = 1;
  for (int b = 0; b < B; ++b) {
    const Seq& s = *seqs[b];
    for (size_t i = 0; i < s.pages.size(); ++i) ptab[b * L.ptable_len + i] = s.pages[i];
    info[4 * b + 0] = s.len;
    info[4 * b + 1] = (s.len + T + SPLIT - 1) / SPLIT;
    splits = std::max(splits, info[4 * b + 1]);
    info[4 * b + 2] = top_k;
    info[4 * b + 3] = dynamic;
    for (int t = 0; t < T; ++t) {
      const int p = s.len + t;   // block row t lands in slot len + t
      slot[b * T + t] = s.pages[p / PAGE] * PAGE + p % PAGE;
    }
  }
  if (c->cap) {
    const ee_model_config& g = c->cfg;
    const size_t need = ee::capture_bytes(g.n_layers, g.d_model, g.n_heads * g.head_dim, g.n_kv_heads * g.head_dim,
                                          g.ffn, g.dtype == EE_BF16 ? ee::DT_BF16 : ee::DT_F32, B * T);
    if (need > c->cap_bytes) return fail(c, EE_EINVAL, "capture buffer too small for this block");
  }
  int rc = order_after_user(c);
  if (rc) return rc;
  ee::Step step{T, B, mode, splits};
  step.cap = c->cap;
  ee::Prof* prof = c->prof.mask ? &c->prof : nullptr;
  // events recorded by graph nodes cannot be timed, and captures are copies
  // of a test aid: profiled or captured blocks run eagerly
  const ee_ctx::Captured* cg = (prof || c->cap || scratch_work) ? nullptr : block_graph(c, step, nullptr);
  if (cg) {
    HIP_TRY(c, hipGraphLaunch(cg->exec, c->st));
    c->prof.used = cg->prof_pairs;
  } else {
    c->prof.used = 0;
    c->prof.overflow = false;
    const hipError_t le = launch_block(c, step, prof, scratch_work ? *scratch_work : c->w);
    if (le != hipSuccess) {
      (void)hipStreamSynchronize(c->st);
      if (c->prof.overflow) return fail(c, EE_EINVAL, "more timed launches in a block than profiling event pairs");
      return hip_fail(c, le, "launch_block");
    }
  }
  HIP_TRY(c, hipStreamSynchronize(c->st));
  for (int i = 0; prof && i < c->prof.used; ++i) {
    float ms = 0.f;
    HIP_TRY(c, hipEventElapsedTime(&ms, c->events[2 * i], c->events[2 * i + 1]));
    c->prof_ms[c->ev_cls[i]] += ms;
    c->prof_n[c->ev_cls[i]] += 1;
  }
  c->last_T = B * T;
  return EE_OK;
}

// Check the draft of one sequence (K tokens, optional parents) before
// anything is staged; fills depth[0..K] for trees.
int check_draft(ee_ctx* c, const int32_t* draft, int K, const int32_t* parent, int* depth) {
  if (K > 0 && !draft) return fail(c, EE_EINVAL, "draft_tokens is NULL");
  for (int i = 0; i < K; ++i)
    if (draft[i] < 0 || draft[i] >= c->cfg.vocab) return fail(c, EE_EINVAL, "draft token outside [0, vocab)");
  if (parent) {
    depth[0] = 0;
    for (int i = 0; i < K; ++i) {
      if (parent[i] < -1 || parent[i] >= i) return fail(c, EE_EINVAL, "parent[i] must be in [-1, i)");
      depth[i + 1] = depth[parent[i] + 1] + 1;
    }
  }
  return EE_OK;
}

// Stage rows b*T .. b*T + T - 1: the pending token and the draft, their
// positions, parent rows and (trees) paths.
void stage_draft(ee_ctx* c, int b, int T, const Seq& s, const int32_t* draft, const int32_t* parent,
                 const int* depth) {
  const Layout& L = c->lay;
  int* tok = reinterpret_cast<int*>(c->h_stage + L.s_tok) + b * T;
  int* pos = reinterpret_cast<int*>(c->h_stage + L.s_pos) + b * T;
  int* prow = reinterpret_cast<int*>(c->h_stage + L.s_prow) + b * T;
  unsigned char* path = c->h_stage + L.s_path + (size_t)b * T * 64;
  tok[0] = s.pending;
  pos[0] = s.len;
  prow[0] = -1;
  for (int r = 1; r < T; ++r) {
    tok[r] = draft[r - 1];
    if (parent) {
      prow[r] = parent[r - 1] + 1;
      pos[r] = s.len + depth[r];
      // the rows on r's path, by depth (attention sees them at n+1 .. n+depth)
      for (int x = r, j = depth[r]; x >= 1; x = prow[x], --j) path[r * 64 + j - 1] = (unsigned char)x;
    } else {
      prow[r] = r - 1;
      pos[r] = s.len + r;
    }
  }
}

// Run rows[0..n) at positions len.. in blocks of at most k_max + 1 rows and
// commit all of them (every row's K/V kept); *last = the greedy token of the
// final row.  On failure the sequence is left as it was.
int commit_rows(ee_ctx* c, Seq& s, const int32_t* rows, int n, int* last) {
  const Layout& L = c->lay;
  int added;
  if (!reserve_pages(c, s, s.len + n, &added)) return fail(c, EE_ECAPACITY, "KV pool exhausted");
  int* tok = reinterpret_cast<int*>(c->h_stage + L.s_tok);
  int* pos = reinterpret_cast<int*>(c->h_stage + L.s_pos);
  int* prow = reinterpret_cast<int*>(c->h_stage + L.s_prow);
  const int len0 = s.len;
  for (int off = 0; off < n; off += L.Tmax) {
    const int T = std::min(L.Tmax, n - off);
    for (int r = 0; r < T; ++r) {
      tok[r] = rows[off + r];
      pos[r] = s.len + r;
      prow[r] = r - 1;
    }
    Seq* one = &s;
    const int rc = run_block(c, &one, 1, T, 0);
    if (rc) {
      s.len = len0;
      unreserve(c, s, added);
      return rc;
    }
    s.len += T;
    *last = c->h_result[1];
  }
  return EE_OK;
}

// One block of n_seq sequences with K draft tokens each: greedy (top_k 0;
// linear, or trees when `parents` is given) or top-k verification (top_k >= 1,
// linear).  Everything is validated and every page reserved before anything
// runs, so an error leaves every sequence as it was.
int verify_many(ee_ctx* c, int n_seq, const int32_t* seqs, const int32_t* drafts, int K, const int32_t* parents,
                int top_k, int dynamic, int32_t* accept_lens, int32_t* next_tokens, int32_t* accepted_nodes,
                int32_t* thresholds) {
  if (!c) return fail(nullptr, EE_EINVAL, "context is NULL");
  if (n_seq < 1 || n_seq > c->cfg.max_seqs) return fail(c, EE_EINVAL, "n_seq outside [1, max_seqs]");
  if (!seqs || !accept_lens || !next_tokens)
    return fail(c, EE_EINVAL, "seqs, accept_lens and next_tokens must be non-NULL");
  if (K < 0 || K > c->cfg.k_max) return fail(c, EE_EINVAL, "K outside [0, k_max]");
  const int T = K + 1;
  if (parents && K > MAX_TREE) return fail(c, EE_EINVAL, "draft trees have at most 64 nodes");
  std::vector<int> depth((size_t)n_seq * (MAX_TREE + 1));
  std::vector<Seq*> ss(n_seq);
  for (int b = 0; b < n_seq; ++b) {
    int rc = check_seq(c, seqs[b]);
    if (rc) return rc;
    for (int b2 = 0; b2 < b; ++b2)
      if (seqs[b2] == seqs[b]) return fail(c, EE_EINVAL, "a sequence appears twice in the batch");
    Seq& s = c->seqs[seqs[b]];
    if (!s.live || s.pending < 0) return fail(c, EE_ESTATE, "verify before prefill");
    if (s.len + T > c->cfg.max_ctx) return fail(c, EE_ECAPACITY, "block would exceed max_ctx");
    if ((rc = check_draft(c, drafts ? drafts + (size_t)b * K : nullptr, K,
                          parents ? parents + (size_t)b * K : nullptr, &depth[(size_t)b * (MAX_TREE + 1)])))
      return rc;
    ss[b] = &s;
  }
  std::vector<int> added(n_seq, 0);
  for (int b = 0; b < n_seq; ++b) {
    if (!reserve_pages(c, *ss[b], ss[b]->len + T, &added[b])) {
      for (int b2 = 0; b2 <= b; ++b2) unreserve(c, *ss[b2], added[b2]);
      return fail(c, EE_ECAPACITY, "KV pool exhausted");
    }
  }
  for (int b = 0; b < n_seq; ++b)
    stage_draft(c, b, T, *ss[b], drafts ? drafts + (size_t)b * K : nullptr,
                parents ? parents + (size_t)b * K : nullptr, &depth[(size_t)b * (MAX_TREE + 1)]);
  const int mode = top_k ? 3 : (parents ? 2 : 1);
  const int rc = run_block(c, ss.data(), n_seq, T, mode, top_k, dynamic);
  if (rc) {
    for (int b = 0; b < n_seq; ++b) unreserve(c, *ss[b], added[b]);
    return rc;
  }
  for (int b = 0; b < n_seq; ++b) {
    const int* res = c->h_result + (size_t)b * c->w.rec;
    const int a = res[0];
    ss[b]->len += 1 + a;
    ss[b]->pending = res[1];
    accept_lens[b] = a;
    next_tokens[b] = res[1];
    if (accepted_nodes)
      for (int i = 0; i < a; ++i) accepted_nodes[(size_t)b * K + i] = res[2 + i] - 1;
    if (thresholds)
      for (int i = 0; i < K; ++i) thresholds[(size_t)b * K + i] = res[2 + i];
  }
  return EE_OK;
}

}  // namespace

extern "C" {

size_t ee_packed_weight_bytes(const ee_model_config* cfg) {
  if (!valid_cfg(cfg, nullptr)) return 0;
  return make_layout(cfg).packed_total;
}

size_t ee_kv_pool_bytes(const ee_model_config* cfg) {
  if (!valid_cfg(cfg, nullptr)) return 0;
  return make_layout(cfg).kv_total;
}

size_t ee_workspace_bytes(const ee_model_config* cfg) {
  if (!valid_cfg(cfg, nullptr)) return 0;
  return make_layout(cfg).ws_total;
}

int32_t ee_create(const ee_model_config* cfg, const ee_weights* wts, void* packed, void* kv_pool,
                  void* workspace, void* hip_stream, ee_ctx** out) {
  std::string why;
  if (!out) return fail(nullptr, EE_EINVAL, "out is NULL");
  *out = nullptr;
  if (!valid_cfg(cfg, &why)) return fail(nullptr, EE_EINVAL, why);
  if (!wts || !packed || !kv_pool || !workspace)
    return fail(nullptr, EE_EINVAL, "weights, packed arena, KV pool and workspace must be non-NULL");
  const int nl = cfg->n_layers;
  if (!wts->embed || !wts->lm_head || !wts->final_gain || !wts->wq || !wts->wk || !wts->wv ||
      !wts->wo || !wts->w_gate || !wts->w_up || !wts->w_down || !wts->attn_gain || !wts->ffn_gain)
    return fail(nullptr, EE_EINVAL, "a weight pointer is NULL");
  for (int l = 0; l < nl; ++l)
    if (!wts->wq[l] || !wts->wk[l] || !wts->wv[l] || !wts->wo[l] || !wts->w_gate[l] ||
        !wts->w_up[l] || !wts->w_down[l] || !wts->attn_gain[l] || !wts->ffn_gain[l])
      return fail(nullptr, EE_EINVAL, "a per-layer weight pointer is NULL");

  ee_ctx* c = new (std::nothrow) ee_ctx();
  if (!c) return fail(nullptr, EE_EINVAL, "out of host memory");
  c->cfg = *cfg;
  c->lay = make_layout(cfg);
  c->user_st = reinterpret_cast<hipStream_t>(hip_stream);
  c->st = c->user_st;   // packing runs on the caller's stream
  c->packed = reinterpret_cast<unsigned char*>(packed);
  c->pool = reinterpret_cast<unsigned char*>(kv_pool);
  c->ws = reinterpret_cast<unsigned char*>(workspace);
  const Layout& L = c->lay;
  const int dt = cfg->dtype == EE_BF16 ? ee::DT_BF16 : ee::DT_F32;
  const size_t esz = ee::esz_of(dt);
  const int d = cfg->d_model, hd = cfg->head_dim, H = cfg->n_heads, Hkv = cfg->n_kv_heads, F = cfg->ffn;

  auto cleanup = [&](int code) {
    if (c->ev_user) (void)hipEventDestroy(c->ev_user);
    if (c->h_stage) (void)hipHostFree(c->h_stage);
    if (c->h_result) (void)hipHostFree(c->h_result);
    g_err = c->err;
    delete c;
    return code;
  };
  hipError_t e;
  if ((e = hipHostMalloc(reinterpret_cast<void**>(&c->h_stage), L.stage_bytes, hipHostMallocDefault)) != hipSuccess ||
      (e = hipHostMalloc(reinterpret_cast<void**>(&c->h_result), (size_t)cfg->max_seqs * (2 + cfg->k_max) * sizeof(int),
                          hipHostMallocDefault)) != hipSuccess) {
    hip_fail(c, e, "hipHostMalloc");
    return cleanup(EE_EHIP);
  }
  memset(c->h_stage, 0, L.stage_bytes);
  if ((e = hipHostGetDevicePointer(reinterpret_cast<void**>(&c->d_stage_src), c->h_stage, 0)) != hipSuccess ||
      (e = hipHostGetDevicePointer(reinterpret_cast<void**>(&c->d_result_dst), c->h_result, 0)) != hipSuccess) {
    hip_fail(c, e, "hipHostGetDevicePointer");
    return cleanup(EE_EHIP);
  }

  // this GPU's static scratch array (ee_verify_noalloc), looked up once per device
  if ((e = hipGetDevice(&c->dev)) != hipSuccess) {
    hip_fail(c, e, "hipGetDevice");
    return cleanup(EE_EHIP);
  }
  {
    void* sp = nullptr;
    if ((e = scratch_address(c->dev, &sp)) != hipSuccess) {
      hip_fail(c, e, "hipGetSymbolAddress(scratch)");
      return cleanup(EE_EHIP);
    }
    c->scratch = reinterpret_cast<unsigned char*>(sp);
  }

  // pack weights
  auto run = [&](hipError_t err, const char* where) {
    if (err != hipSuccess) { hip_fail(c, err, where); return false; }
    return true;
  };
  bool ok = run(ee::launch_copy(wts->embed, c->packed + L.embed, (size_t)cfg->vocab * d * esz, c->st), "copy embed") &&
            run(ee::launch_copy(wts->final_gain, c->packed + L.final_gain, (size_t)d * 4, c->st), "copy gain");
  ee::PackSrc ps{wts->lm_head, cfg->vocab, 0};
  ok = ok && run(ee::launch_pack(ps, c->packed + L.lm_head, d, dt, c->st), "pack lm_head");
  c->layers.resize(nl);
  for (int l = 0; l < nl && ok; ++l) {
    unsigned char* lb = c->packed + L.layers0 + (size_t)l * L.per_layer;
    ee::LayerPtrs& lp = c->layers[l];
    lp.wqkv = reinterpret_cast<const uint4*>(lb + L.l_wqkv);
    lp.wo = reinterpret_cast<const uint4*>(lb + L.l_wo);
    lp.wgu = reinterpret_cast<const uint4*>(lb + L.l_wgu);
    lp.wd = reinterpret_cast<const uint4*>(lb + L.l_wd);
    lp.attn_gain = reinterpret_cast<const float*>(lb + L.l_again);
    lp.ffn_gain = reinterpret_cast<const float*>(lb + L.l_fgain);
    const ee::PackSrc parts[] = {
        {wts->wq[l], H * hd, 0}, {wts->wk[l], Hkv * hd, H * hd}, {wts->wv[l], Hkv * hd, (H + Hkv) * hd}};
    for (const auto& p : parts) ok = ok && run(ee::launch_pack(p, lb + L.l_wqkv, d, dt, c->st), "pack wqkv");
    ok = ok && run(ee::launch_pack({wts->wo[l], d, 0}, lb + L.l_wo, H * hd, dt, c->st), "pack wo");
    ok = ok && run(ee::launch_pack({wts->w_gate[l], F, 0}, lb + L.l_wgu, d, dt, c->st), "pack w_gate");
    ok = ok && run(ee::launch_pack({wts->w_up[l], F, F}, lb + L.l_wgu, d, dt, c->st), "pack w_up");
    ok = ok && run(ee::launch_pack({wts->w_down[l], d, 0}, lb + L.l_wd, F, dt, c->st), "pack w_down");
    ok = ok && run(ee::launch_copy(wts->attn_gain[l], lb + L.l_again, (size_t)d * 4, c->st), "copy gain") &&
         run(ee::launch_copy(wts->ffn_gain[l], lb + L.l_fgain, (size_t)d * 4, c->st), "copy gain");
  }
  // rotary table (cos, sin) of every position, computed in double
  std::vector<float> rope((size_t)cfg->max_ctx * hd);
  for (int p = 0; p < cfg->max_ctx; ++p)
    for (int i = 0; i < hd / 2; ++i) {
      const double ang = (double)p * pow((double)cfg->rope_theta, -2.0 * i / hd);
      rope[((size_t)p * (hd / 2) + i) * 2 + 0] = (float)cos(ang);
      rope[((size_t)p * (hd / 2) + i) * 2 + 1] = (float)sin(ang);
    }
  ok = ok && run(hipMemcpyAsync(c->ws + L.rope, rope.data(), rope.size() * 4, hipMemcpyHostToDevice, c->st), "upload rope");
  ok = ok && run(hipMemsetAsync(c->pool, 0, L.kv_total, c->st), "zero KV pool");
  ok = ok && run(hipStreamSynchronize(c->st), "hipStreamSynchronize");
  if (!ok) return cleanup(EE_EHIP);
  // every later call runs on a library stream (capturable; the legacy default
  // stream is not), ordered after the caller's stream at the start of a call
  hipStream_t own = nullptr;
  if (!run(hipStreamCreateWithFlags(&own, hipStreamNonBlocking), "hipStreamCreate") ||
      !run(hipEventCreateWithFlags(&c->ev_user, hipEventDisableTiming), "hipEventCreate")) {
    if (own) (void)hipStreamDestroy(own);
    return cleanup(EE_EHIP);
  }
  c->st = own;

  ee::Model& m = c->m;
  m.L = nl; m.d = d; m.H = H; m.Hkv = Hkv; m.hd = hd; m.F = F; m.V = cfg->vocab; m.dt = dt;
  m.eps = cfg->rms_eps; m.max_ctx = cfg->max_ctx; m.max_pages = L.n_pages;
  m.embed = c->packed + L.embed;
  m.lm_head = reinterpret_cast<const uint4*>(c->packed + L.lm_head);
  m.final_gain = reinterpret_cast<const float*>(c->packed + L.final_gain);
  m.layers = c->layers.data();
  m.kv_pool = c->pool;
  m.rope = reinterpret_cast<const float2*>(c->ws + L.rope);
  bind_work(c);
  c->seqs.assign(cfg->max_seqs, Seq());
  c->free_pages.clear();
  for (int p = L.n_pages - 1; p >= 0; --p) c->free_pages.push_back(p);
  *out = c;
  return EE_OK;
}

int32_t ee_destroy(ee_ctx* c) {
  if (!c) return fail(nullptr, EE_EINVAL, "context is NULL");
  if (c->st) (void)hipStreamSynchronize(c->st);
  for (auto& kv : c->graphs) (void)hipGraphExecDestroy(kv.second.exec);
  for (hipEvent_t e : c->events) (void)hipEventDestroy(e);
  if (c->ev_user) (void)hipEventDestroy(c->ev_user);
  if (c->st && c->st != c->user_st) (void)hipStreamDestroy(c->st);
  if (c->h_stage) (void)hipHostFree(c->h_stage);
  if (c->h_result) (void)hipHostFree(c->h_result);
  delete c;
  return EE_OK;
}

int32_t ee_prefill(ee_ctx* c, int32_t seq, const int32_t* tokens, int32_t n, int32_t* next_token) {
  int rc = check_seq(c, seq);
  if (rc) return rc;
  if (!tokens || !next_token) return fail(c, EE_EINVAL, "tokens and next_token must be non-NULL");
  if (n < 1) return fail(c, EE_EINVAL, "prefill needs at least one token");
  Seq& s = c->seqs[seq];
  if (s.live) return fail(c, EE_ESTATE, "sequence already holds tokens (roll it back to 0 first)");
  if (n > c->cfg.max_ctx - 1) return fail(c, EE_ECAPACITY, "prompt longer than max_ctx - 1");
  for (int i = 0; i < n; ++i)
    if (tokens[i] < 0 || tokens[i] >= c->cfg.vocab) return fail(c, EE_EINVAL, "token outside [0, vocab)");
  int last;
  if ((rc = commit_rows(c, s, tokens, n, &last))) return rc;
  s.live = true;
  s.pending = last;
  *next_token = last;
  return EE_OK;
}

int32_t ee_extend(ee_ctx* c, int32_t seq, const int32_t* tokens, int32_t n, int32_t* next_token) {
  int rc = check_seq(c, seq);
  if (rc) return rc;
  if ((n > 0 && !tokens) || !next_token) return fail(c, EE_EINVAL, "tokens and next_token must be non-NULL");
  if (n < 0) return fail(c, EE_EINVAL, "n must be >= 0");
  Seq& s = c->seqs[seq];
  if (!s.live || s.pending < 0) return fail(c, EE_ESTATE, "extend before prefill");
  for (int i = 0; i < n; ++i)
    if (tokens[i] < 0 || tokens[i] >= c->cfg.vocab) return fail(c, EE_EINVAL, "token outside [0, vocab)");
  if ((size_t)s.len + n + 2 > (size_t)c->cfg.max_ctx) return fail(c, EE_ECAPACITY, "sequence would exceed max_ctx");
  std::vector<int32_t> rows((size_t)n + 1);
  rows[0] = s.pending;
  for (int i = 0; i < n; ++i) rows[i + 1] = tokens[i];
  int last;
  if ((rc = commit_rows(c, s, rows.data(), n + 1, &last))) return rc;
  s.pending = last;
  *next_token = last;
  return EE_OK;
}

int32_t ee_verify(ee_ctx* c, int32_t seq, const int32_t* draft, int32_t K, const int32_t* parent,
                  int32_t* accept_len, int32_t* next_token, int32_t* accepted_nodes) {
  int rc = check_seq(c, seq);
  if (rc) return rc;
  if (!accept_len || !next_token) return fail(c, EE_EINVAL, "accept_len and next_token must be non-NULL");
  Seq& s = c->seqs[seq];
  if (!s.live || s.pending < 0) return fail(c, EE_ESTATE, "verify before prefill");
  if (K < 0 || K > c->cfg.k_max) return fail(c, EE_EINVAL, "K outside [0, k_max]");
  if (parent && K > MAX_TREE) return fail(c, EE_EINVAL, "draft trees have at most 64 nodes");
  int depth[MAX_TREE + 1];
  if ((rc = check_draft(c, draft, K, parent, depth))) return rc;
  const int T = K + 1;
  if (s.len + T > c->cfg.max_ctx) return fail(c, EE_ECAPACITY, "block would exceed max_ctx");
  int added;
  if (!reserve_pages(c, s, s.len + T, &added)) return fail(c, EE_ECAPACITY, "KV pool exhausted");
  stage_draft(c, 0, T, s, draft, parent, depth);
  Seq* one = &s;
  rc = run_block(c, &one, 1, T, parent ? 2 : 1);
  if (rc) {
    unreserve(c, s, added);
    return rc;
  }
  const int a = c->h_result[0];
  s.len += 1 + a;
  s.pending = c->h_result[1];
  *accept_len = a;
  *next_token = s.pending;
  if (accepted_nodes)
    for (int i = 0; i < a; ++i) accepted_nodes[i] = c->h_result[2 + i] - 1;
  return EE_OK;
}

int32_t ee_verify_noalloc(ee_ctx* c, int32_t seq, const int32_t* draft, int32_t K, const int32_t* parent,
                          int32_t* accept_len, int32_t* next_token, int32_t* accepted_nodes) {
  int rc = check_seq(c, seq);
  if (rc) return rc;
  if (!accept_len || !next_token) return fail(c, EE_EINVAL, "accept_len and next_token must be non-NULL");
  Seq& s = c->seqs[seq];
  if (!s.live || s.pending < 0) return fail(c, EE_ESTATE, "verify before prefill");
  if (K < 0 || K > c->cfg.k_max) return fail(c, EE_EINVAL, "K outside [0, k_max]");
  if (parent && K > MAX_TREE) return fail(c, EE_EINVAL, "draft trees have at most 64 nodes");
  int depth[MAX_TREE + 1];
  if ((rc = check_draft(c, draft, K, parent, depth))) return rc;
  const int T = K + 1;
  if (s.len + T > c->cfg.max_ctx) return fail(c, EE_ECAPACITY, "block would exceed max_ctx");
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != c->dev)
    return fail(c, EE_EINVAL, "the context's GPU must be the current device");
  // scratch of this block: attention split states, then GEMM slice partials
  const ee_model_config& g = c->cfg;
  const size_t splits = (size_t)(s.len + T + SPLIT - 1) / SPLIT;
  const size_t attn = up(splits * g.n_kv_heads * (size_t)T * (g.n_heads / g.n_kv_heads) * (g.head_dim + 2) * 4);
  const size_t part = up(partial_cols(g) * (size_t)T * 4);
  if (attn + part > NOALLOC_SCRATCH_BYTES)
    return fail(c, EE_ECAPACITY, "this block needs " + std::to_string(attn + part) +
                                     " bytes of scratch, more than the 16 MiB static buffer of ee_verify_noalloc");
  int added;
  if (!reserve_pages(c, s, s.len + T, &added)) return fail(c, EE_ECAPACITY, "KV pool exhausted");
  stage_draft(c, 0, T, s, draft, parent, depth);
  ee::Work w = c->w;
  w.attn_part = reinterpret_cast<float*>(c->scratch);
  w.part = reinterpret_cast<float*>(c->scratch + attn);
  Seq* one = &s;
  rc = run_block(c, &one, 1, T, parent ? 2 : 1, 0, 0, &w);
  if (rc) {
    unreserve(c, s, added);
    return rc;
  }
  const int a = c->h_result[0];
  s.len += 1 + a;
  s.pending = c->h_result[1];
  *accept_len = a;
  *next_token = s.pending;
  if (accepted_nodes)
    for (int i = 0; i < a; ++i) accepted_nodes[i] = c->h_result[2 + i] - 1;
  return EE_OK;
}

int32_t ee_verify_batch(ee_ctx* c, int32_t n_seq, const int32_t* seqs, const int32_t* drafts, int32_t K,
                        const int32_t* parents, int32_t* accept_lens, int32_t* next_tokens,
                        int32_t* accepted_nodes) {
  return verify_many(c, n_seq, seqs, drafts, K, parents, 0, 0, accept_lens, next_tokens, accepted_nodes, nullptr);
}

int32_t ee_verify_topk(ee_ctx* c, int32_t n_seq, const int32_t* seqs, const int32_t* drafts, int32_t K,
                       int32_t top_k, int32_t dynamic, int32_t* accept_lens, int32_t* next_tokens,
                       int32_t* thresholds) {
  if (!c) return fail(nullptr, EE_EINVAL, "context is NULL");
  if (top_k < 1 || top_k > 8 || top_k > c->cfg.vocab) return fail(c, EE_EINVAL, "top_k outside [1, min(8, vocab)]");
  return verify_many(c, n_seq, seqs, drafts, K, nullptr, top_k, dynamic ? 1 : 0, accept_lens, next_tokens,
                     nullptr, thresholds);
}

int32_t ee_verify_sample(ee_ctx* c, int32_t seq, const int32_t* draft, int32_t K, const float* q_dev,
                         const float* eps, const float* u, float temperature, int32_t residual,
                         int32_t* accept_len, int32_t* next_token) {
  int rc = check_seq(c, seq);
  if (rc) return rc;
  if (!accept_len || !next_token || !u || (K > 0 && !eps))
    return fail(c, EE_EINVAL, "eps (K > 0), u, accept_len and next_token must be non-NULL");
  Seq& s = c->seqs[seq];
  if (!s.live || s.pending < 0) return fail(c, EE_ESTATE, "verify before prefill");
  if (K < 0 || K > c->cfg.k_max) return fail(c, EE_EINVAL, "K outside [0, k_max]");
  if (!(temperature > 0.f) || !(temperature < INFINITY)) return fail(c, EE_EINVAL, "temperature must be positive");
  if (c->cfg.vocab > 4096 * 64) return fail(c, EE_EINVAL, "stochastic verification handles vocabularies up to 262144");
  for (int i = 0; i < K; ++i)
    if (!(eps[i] >= 0.f && eps[i] < 1.f)) return fail(c, EE_EINVAL, "eps outside [0, 1)");
  for (int i = 0; i <= K; ++i)
    if (!(u[i] >= 0.f && u[i] < 1.f)) return fail(c, EE_EINVAL, "u outside [0, 1)");
  int depth[1];
  if ((rc = check_draft(c, draft, K, nullptr, depth))) return rc;
  const int T = K + 1;
  if (s.len + T > c->cfg.max_ctx) return fail(c, EE_ECAPACITY, "block would exceed max_ctx");
  int added;
  if (!reserve_pages(c, s, s.len + T, &added)) return fail(c, EE_ECAPACITY, "KV pool exhausted");
  stage_draft(c, 0, T, s, draft, nullptr, depth);
  const Layout& L = c->lay;
  float* se = reinterpret_cast<float*>(c->h_stage + L.s_eps);
  float* su = reinterpret_cast<float*>(c->h_stage + L.s_unif);
  for (int i = 0; i < K; ++i) se[i] = eps[i];
  for (int i = 0; i <= K; ++i) su[i] = u[i];
  struct {
    unsigned long long q;
    float temperature;
    int32_t residual;
  } sp{(unsigned long long)(uintptr_t)q_dev, temperature, residual ? 1 : 0};
  static_assert(sizeof(sp) == 16, "staged sampling parameters");
  memcpy(c->h_stage + L.s_sparam, &sp, sizeof sp);
  Seq* one = &s;
  rc = run_block(c, &one, 1, T, 4);
  if (rc) {
    unreserve(c, s, added);
    return rc;
  }
  const int a = c->h_result[0];
  s.len += 1 + a;
  s.pending = c->h_result[1];
  *accept_len = a;
  *next_token = s.pending;
  return EE_OK;
}

int32_t ee_kv_rollback(ee_ctx* c, int32_t seq, int32_t new_len, int32_t pending_token) {
  int rc = check_seq(c, seq);
  if (rc) return rc;
  Seq& s = c->seqs[seq];
  if (new_len < 0) return fail(c, EE_EINVAL, "new_len must be >= 0");
  if (new_len > s.len) return fail(c, EE_ESTATE, "rollback beyond the committed length");
  if (new_len == 0 && pending_token == -1) {
    unreserve(c, s, (int)s.pages.size());
    s = Seq();
    return EE_OK;
  }
  if (pending_token < 0 || pending_token >= c->cfg.vocab)
    return fail(c, EE_EINVAL, "pending_token outside [0, vocab)");
  if (!s.live) return fail(c, EE_ESTATE, "sequence is empty");
  const int keep = (new_len + PAGE - 1) / PAGE;
  unreserve(c, s, (int)s.pages.size() - keep);
  s.len = new_len;
  s.pending = pending_token;
  return EE_OK;
}

int32_t ee_seq_state(ee_ctx* c, int32_t seq, int32_t* len, int32_t* pending_token) {
  int rc = check_seq(c, seq);
  if (rc) return rc;
  if (!len || !pending_token) return fail(c, EE_EINVAL, "outputs must be non-NULL");
  *len = c->seqs[seq].len;
  *pending_token = c->seqs[seq].live ? c->seqs[seq].pending : -1;
  return EE_OK;
}

int32_t ee_get_logits(ee_ctx* c, float* host_out, int32_t rows) {
  if (!c) return fail(nullptr, EE_EINVAL, "context is NULL");
  if (!host_out) return fail(c, EE_EINVAL, "host_out is NULL");
  if (c->last_T == 0) return fail(c, EE_ESTATE, "no block has run yet");
  if (rows != c->last_T) return fail(c, EE_EINVAL, "rows must equal the last block's row count");
  HIP_TRY(c, hipMemcpyAsync(host_out, c->w.logits, (size_t)rows * c->cfg.vocab * 4, hipMemcpyDeviceToHost, c->st));
  HIP_TRY(c, hipStreamSynchronize(c->st));
  return EE_OK;
}

int32_t ee_read_kv(ee_ctx* c, int32_t seq, int32_t layer, void* host_k, void* host_v) {
  int rc = check_seq(c, seq);
  if (rc) return rc;
  if (layer < 0 || layer >= c->cfg.n_layers) return fail(c, EE_EINVAL, "layer out of range");
  const Seq& s = c->seqs[seq];
  const size_t esz = c->cfg.dtype == EE_BF16 ? 2 : 4;
  const int Hkv = c->cfg.n_kv_heads, hd = c->cfg.head_dim;
  const size_t blk = (size_t)PAGE * hd * esz;            // one (page, kv, head) block
  std::vector<unsigned char> page(2 * Hkv * blk);
  for (size_t pi = 0; pi * PAGE < (size_t)s.len; ++pi) {
    const unsigned char* src = c->pool + layer * c->lay.kv_layer + (size_t)s.pages[pi] * 2 * Hkv * blk;
    HIP_TRY(c, hipMemcpyAsync(page.data(), src, page.size(), hipMemcpyDeviceToHost, c->st));
    HIP_TRY(c, hipStreamSynchronize(c->st));
    for (int sp = 0; sp < PAGE && (int)(pi * PAGE) + sp < s.len; ++sp) {
      const size_t slot = pi * PAGE + sp;
      for (int g = 0; g < Hkv; ++g)
        for (int dim = 0; dim < hd; ++dim) {
          const size_t dst = ((slot * Hkv + g) * hd + dim) * esz;
          if (host_k)
            memcpy(reinterpret_cast<unsigned char*>(host_k) + dst,
                   page.data() + (0 * Hkv + g) * blk + ((size_t)sp * hd + dim) * esz, esz);
          if (host_v)
            memcpy(reinterpret_cast<unsigned char*>(host_v) + dst,
                   page.data() + (1 * Hkv + g) * blk + ((size_t)dim * PAGE + sp) * esz, esz);
        }
    }
  }
  return EE_OK;
}

int32_t ee_load_kv(ee_ctx* c, int32_t seq, int32_t n, int32_t pending, const void* host_k, const void* host_v) {
  int rc = check_seq(c, seq);
  if (rc) return rc;
  if (!host_k || !host_v) return fail(c, EE_EINVAL, "host_k and host_v must be non-NULL");
  if (n < 1) return fail(c, EE_EINVAL, "n must be >= 1");
  if (pending < 0 || pending >= c->cfg.vocab) return fail(c, EE_EINVAL, "pending token outside [0, vocab)");
  Seq& s = c->seqs[seq];
  if (s.live) return fail(c, EE_ESTATE, "sequence already holds tokens (roll it back to 0 first)");
  if (n > c->cfg.max_ctx - 1) return fail(c, EE_ECAPACITY, "cache longer than max_ctx - 1");
  if ((rc = order_after_user(c))) return rc;
  int added;
  if (!reserve_pages(c, s, n, &added)) return fail(c, EE_ECAPACITY, "KV pool exhausted");
  const size_t esz = c->cfg.dtype == EE_BF16 ? 2 : 4;
  const int Hkv = c->cfg.n_kv_heads, hd = c->cfg.head_dim;
  const size_t blk = (size_t)PAGE * hd * esz;            // one (page, kv, head) block
  const size_t layer_in = (size_t)n * Hkv * hd * esz;     // one layer of host_k / host_v
  std::vector<unsigned char> page(2 * Hkv * blk);
  for (int layer = 0; layer < c->cfg.n_layers; ++layer)
    for (size_t pi = 0; pi < s.pages.size(); ++pi) {
      // K rows [slot][dim] and V^T [dim][slot] of this page; slots past n stay zero
      std::fill(page.begin(), page.end(), 0);
      for (int sp = 0; sp < PAGE && (int)(pi * PAGE) + sp < n; ++sp) {
        const size_t slot = pi * PAGE + sp;
        for (int g = 0; g < Hkv; ++g)
          for (int dim = 0; dim < hd; ++dim) {
            const size_t src = layer * layer_in + ((slot * Hkv + g) * hd + dim) * esz;
            memcpy(page.data() + (0 * Hkv + g) * blk + ((size_t)sp * hd + dim) * esz,
                   reinterpret_cast<const unsigned char*>(host_k) + src, esz);
            memcpy(page.data() + (1 * Hkv + g) * blk + ((size_t)dim * PAGE + sp) * esz,
                   reinterpret_cast<const unsigned char*>(host_v) + src, esz);
          }
      }
      unsigned char* dst = c->pool + layer * c->lay.kv_layer + (size_t)s.pages[pi] * 2 * Hkv * blk;
      hipError_t e = hipMemcpyAsync(dst, page.data(), page.size(), hipMemcpyHostToDevice, c->st);
      if (e == hipSuccess) e = hipStreamSynchronize(c->st);   // the page buffer is refilled next
      if (e != hipSuccess) {
        unreserve(c, s, added);
        return hip_fail(c, e, "hipMemcpy");
      }
    }
  s.len = n;
  s.live = true;
  s.pending = pending;
  return EE_OK;
}

size_t ee_capture_bytes(const ee_model_config* cfg, int32_t rows) {
  if (!valid_cfg(cfg, nullptr) || rows < 1) return 0;
  return ee::capture_bytes(cfg->n_layers, cfg->d_model, cfg->n_heads * cfg->head_dim, cfg->n_kv_heads * cfg->head_dim,
                           cfg->ffn, cfg->dtype == EE_BF16 ? ee::DT_BF16 : ee::DT_F32, rows);
}

int32_t ee_capture(ee_ctx* c, void* dev_buf, size_t bytes) {
  if (!c) return fail(nullptr, EE_EINVAL, "context is NULL");
  if (dev_buf && bytes == 0) return fail(c, EE_EINVAL, "a capture buffer needs a size");
  c->cap = reinterpret_cast<unsigned char*>(dev_buf);
  c->cap_bytes = dev_buf ? bytes : 0;
  return EE_OK;
}

int32_t ee_use_graphs(ee_ctx* c, int32_t on) {
  if (!c) return fail(nullptr, EE_EINVAL, "context is NULL");
  c->graphs_on = on != 0;
  return EE_OK;
}

int32_t ee_profile(ee_ctx* c, uint32_t class_mask) {
  if (!c) return fail(nullptr, EE_EINVAL, "context is NULL");
  if (class_mask >> ee::PC_N) return fail(c, EE_EINVAL, "unknown profiling class");
  if (class_mask && c->events.empty()) {
    // enough pairs for every timed launch of one block
    const int pairs = ee::prof_pairs_per_block(c->cfg.n_layers);
    c->events.resize(2 * pairs);
    for (auto& e : c->events) {
      hipError_t r = hipEventCreate(&e);
      if (r != hipSuccess) return hip_fail(c, r, "hipEventCreate");
    }
    c->ev_cls.assign(pairs, 0);
    c->prof.ev = c->events.data();
    c->prof.cls = c->ev_cls.data();
    c->prof.cap = pairs;
  }
  c->prof.mask = class_mask;
  return EE_OK;
}

int32_t ee_profile_read(ee_ctx* c, double* ms, int64_t* launches, int32_t reset) {
  if (!c) return fail(nullptr, EE_EINVAL, "context is NULL");
  for (int i = 0; i < ee::PC_N; ++i) {
    if (ms) ms[i] = c->prof_ms[i];
    if (launches) launches[i] = c->prof_n[i];
    if (reset) {
      c->prof_ms[i] = 0.0;
      c->prof_n[i] = 0;
    }
  }
  return EE_OK;
}

int32_t ee_time_gemm(ee_ctx* c, uint32_t cls, int32_t rows, int32_t reps, double* us_per_launch) {
  if (!c) return fail(nullptr, EE_EINVAL, "context is NULL");
  if (!us_per_launch || reps < 1) return fail(c, EE_EINVAL, "us_per_launch must be non-NULL and reps >= 1");
  if (cls != EE_PROF_QKV && cls != EE_PROF_OPROJ && cls != EE_PROF_GATEUP && cls != EE_PROF_DOWN &&
      cls != EE_PROF_LMHEAD)
    return fail(c, EE_EINVAL, "class must be one of the four projections or the LM head");
  if (rows < 1 || rows > c->lay.Rmax) return fail(c, EE_EINVAL, "rows outside [1, max_seqs * (k_max + 1)]");
  hipEvent_t e0 = nullptr, e1 = nullptr;
  HIP_TRY(c, hipEventCreate(&e0));
  if (hipEventCreate(&e1) != hipSuccess) {
    (void)hipEventDestroy(e0);
    return fail(c, EE_EHIP, "hipEventCreate");
  }
  hipError_t e = hipEventRecord(e0, c->st);
  for (int r = 0; r < reps && e == hipSuccess; ++r) e = ee::run_gemm_sequence(c->m, c->w, (int)cls, rows, c->st);
  if (e == hipSuccess) e = hipEventRecord(e1, c->st);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (e != hipSuccess) return hip_fail(c, e, "ee_time_gemm");
  *us_per_launch = (double)ms * 1e3 / ((double)reps * c->cfg.n_layers);
  return EE_OK;
}

int32_t ee_time_stream_read(ee_ctx* c, const void* dev_buf, size_t bytes, int32_t reps, double* us_per_pass) {
  if (!c) return fail(nullptr, EE_EINVAL, "context is NULL");
  if (!dev_buf || !us_per_pass || reps < 1 || bytes < ((size_t)256 << 10) || bytes % 16)
    return fail(c, EE_EINVAL, "a buffer of at least 256 KiB (a multiple of 16 bytes), reps >= 1 and an output are needed");
  hipEvent_t e0 = nullptr, e1 = nullptr;
  HIP_TRY(c, hipEventCreate(&e0));
  if (hipEventCreate(&e1) != hipSuccess) {
    (void)hipEventDestroy(e0);
    return fail(c, EE_EHIP, "hipEventCreate");
  }
  unsigned* sink = reinterpret_cast<unsigned*>(c->w.greedy);
  hipError_t e = ee::run_stream_read(dev_buf, bytes, sink, c->st);   // warm-up pass
  if (e == hipSuccess) e = hipEventRecord(e0, c->st);
  for (int r = 0; r < reps && e == hipSuccess; ++r) e = ee::run_stream_read(dev_buf, bytes, sink, c->st);
  if (e == hipSuccess) e = hipEventRecord(e1, c->st);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (e != hipSuccess) return hip_fail(c, e, "ee_time_stream_read");
  *us_per_pass = (double)ms * 1e3 / reps;
  return EE_OK;
}

const char* ee_last_error(const ee_ctx* c) { return c ? c->err.c_str() : g_err.c_str(); }

}  // extern "C"
