// kf_api.cpp -- C ABI of the K-Forcing decode library (include/kforcing.h).
//
// Host side: argument validation, the per-context sequence state machine, the
// device memory plan inside the caller's state buffer, weight packing, and the
// kernel sequence of one step (paper Appendix C.1: embed real rows and noise
// rows, L pre-norm Transformer blocks over the cached context, final norm,
// tied head, token selection, commit of the real rows' K/V).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <functional>
#include <mutex>
#include <string>
#include <vector>

#include "kforcing.h"
#include "kf_internal.h"

namespace {

constexpr int32_t kMagic = 0x4B465731;
constexpr int kHeaderInts = 16;
constexpr int32_t kBlobTemperature = 1;  // header word 9: temperature encoder present
constexpr int32_t kBlobRmsRope = 2;      // header word 9: RMSNorm + rotary positions

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Attention key-split workspace: partial states for up to 8192 (sequence,
// head, query row, split) entries (the launcher splits only grids of fewer
// than 256 workgroups, into at most 512 in total).
constexpr int kAttnEntries = 8192;
// Split-K GEMM workspace (fp32 parts of the plain GEMMs of small steps).
constexpr size_t kSplitBytes = (size_t)8 << 20;
// Captured served steps kept per context (one per (sequences, pending, k)).
constexpr size_t kServeGraphs = 16;
// Rows per sampling-head chunk of kf_teacher_targets: the head partials of a
// chunk take rows * (Vpad / 128) * 36 bytes (about 116 MB at vocabulary 50257).
constexpr int kTeacherChunk = 8192;
// Noise rows computed ahead per chunk of generate passes (kf_generate): at
// least this many rows per chunk, or one pass of the largest batch.
constexpr int kNoiseAheadRows = 8192;

// ------------------------------------------------------------ memory plan
struct LayerOff {
  size_t ln1_g, ln1_b, wqkv, bqkv, wo, bo, ln2_g, ln2_b, w1, b1, w2, b2;
  size_t qkv_c1, qkv_c2, up_c1, up_c2;  // folded LayerNorm sums (fp32)
};

struct Plan {
  int es = 0;        // bytes per element of the compute dtype
  int Vpad = 0;      // vocabulary rounded up to 256 (padding rows are zero)
  int n_tiles = 0;   // head column tiles
  int rows_max = 0;  // largest number of rows in one step
  int head_max = 0;  // largest number of head rows in one step
  int logit_rows = 0;
  size_t wbegin = 0, wend = 0;
  size_t tok = 0, pos = 0, nw1 = 0, nb1 = 0, nw2 = 0, nb2 = 0, omega = 0, lnf_g = 0, lnf_b = 0;
  size_t head_c1 = 0, head_c2 = 0, head_w = 0;  // folded final norm; gain-scaled token table
  size_t tw1 = 0, tb1 = 0, tw2 = 0, tb2 = 0;     // temperature encoder (KF_FLAG_TEMPERATURE)
  size_t rope = 0;                              // rotary table [n_ctx][d_rot/2] (KF_FLAG_RMS_ROPE)
  size_t temb = 0;                              // per-sequence temperature embedding [max_batch][d]
  std::vector<LayerOff> layer;
  int Tp = 0;           // per-sequence KV capacity rounded up to whole pages
  int npp = 0;          // pages per sequence (Tp / kPage)
  int n_pages = 0;      // pages in the KV pool
  size_t page_bytes = 0;
  size_t kv = 0, kv_bytes = 0;
  size_t meta = 0;      // continuous batching: slot map [max_batch], committed lengths
                        // [max_batch], page table [max_batch][npp] (int32)
  size_t serve_noise = 0, serve_out = 0;  // fixed [max_batch][max_k] buffers of graph-replayed steps
  size_t X = 0, Xh = 0, lnst = 0, A = 0, Q = 0, O = 0, Hm = 0, noise = 0, pval = 0, pidx = 0;
  size_t logits = 0, dstate = 0, pend = 0;
  int teacher_rows = 0;                    // rows per sampling-head chunk (KF_FLAG_TEACHER)
  size_t roll_kv = 0;                      // per-layer K/V of the teacher rollout (KF_FLAG_ROLLOUT)
  size_t tmax = 0, tsub = 0;               // sampling-head partials of one chunk
  size_t att_m = 0, att_l = 0, att_o = 0;  // attention key-split partial states
  size_t split_part = 0;                   // split-K GEMM parts
  int nz_rows = 0;                         // noise rows computed ahead: capacity
  size_t nzA = 0, nzH = 0, nz = 0;         // their sinusoids, hidden layer, output (fp32)
  size_t total = 0;
};

bool config_ok(const kf_config& c, std::string* why) {
  auto bad = [&](const char* m) {
    if (why) *why = m;
    return false;
  };
  if (c.n_layer < 1) return bad("n_layer must be >= 1");
  if (c.d_model < 64 || c.d_model % 64) return bad("d_model must be a positive multiple of 64");
  if (c.d_model > 2048) return bad("d_model must be <= 2048");
  if (c.n_head < 1 || c.d_model % c.n_head) return bad("n_head must divide d_model");
  int dh = c.d_model / c.n_head;
  if (dh != 32 && dh != 64 && dh != 128) return bad("d_model / n_head must be 32, 64 or 128");
  if (c.d_mlp < 64 || c.d_mlp % 64) return bad("d_mlp must be a positive multiple of 64");
  if (c.vocab < 2) return bad("vocab must be >= 2");
  if (c.n_ctx < 8 || c.n_ctx % 8) return bad("n_ctx must be a positive multiple of 8");
  if (c.dtype != KF_FP32 && c.dtype != KF_BF16) return bad("dtype must be KF_FP32 or KF_BF16");
  if (c.max_batch < 1 || c.max_batch > 65535) return bad("max_batch must be in [1, 65535]");
  if (c.max_k < 1 || c.max_k > c.n_ctx) return bad("max_k must be in [1, n_ctx]");
  if (c.max_prompt < 1 || c.max_prompt > c.n_ctx) return bad("max_prompt must be in [1, n_ctx]");
  if (c.flags & ~(KF_FLAG_DEBUG_LOGITS | KF_FLAG_TEMPERATURE | KF_FLAG_TEACHER | KF_FLAG_ROLLOUT |
                  KF_FLAG_RMS_ROPE | KF_FLAG_SERVING))
    return bad("unknown flag bits");
  if (c.kv_pages < 0) return bad("kv_pages must be >= 0");
  if (c.kv_pages > 0 && !(c.flags & KF_FLAG_SERVING)) return bad("kv_pages needs KF_FLAG_SERVING");
  if ((long long)c.max_batch * ((c.n_ctx + kPage - 1) / kPage) > (1 << 24))
    return bad("max_batch * pages per sequence must stay below 2^24");
  // GEMM operands are addressed through buffer descriptors with 32-bit byte
  // ranges: the largest activation matrix of a step must stay below 2 GiB.
  const long long es = c.dtype == KF_BF16 ? 2 : 4;
  long long rows = (long long)c.max_batch * ((c.max_prompt > c.max_k ? c.max_prompt : c.max_k) + c.max_k);
  if (c.flags & KF_FLAG_ROLLOUT) {
    const long long r2 = 2LL * c.max_batch * c.max_prompt * c.max_k;  // DoubleForward rows
    if (r2 > rows) rows = r2;
  }
  const long long width = c.d_mlp > 4 * c.d_model ? c.d_mlp : 4 * c.d_model;
  if (rows * width * es >= (1LL << 31) || rows * c.d_model * 4 >= (1LL << 31))
    return bad("max_batch * (max(max_prompt, max_k) + max_k) rows too large for one step");
  return true;
}

void make_plan(const kf_config& c, Plan& p) {
  const size_t d = c.d_model, f = c.d_mlp, T = c.n_ctx, L = c.n_layer;
  p.es = c.dtype == KF_BF16 ? 2 : 4;
  p.Vpad = (c.vocab + 255) / 256 * 256;
  p.n_tiles = p.Vpad / kf::kHeadTileN;
  p.rows_max = c.max_batch * ((c.max_prompt > c.max_k ? c.max_prompt : c.max_k) + c.max_k);
  p.head_max = c.max_batch * c.max_k;
  if (c.flags & KF_FLAG_ROLLOUT) {
    const int r2 = 2 * c.max_batch * c.max_prompt * c.max_k;
    if (r2 > p.rows_max) p.rows_max = r2;
    if (c.max_batch * c.max_prompt * c.max_k > p.head_max) p.head_max = c.max_batch * c.max_prompt * c.max_k;
  }
  if (c.flags & KF_FLAG_TEACHER) {
    const long long tr = (long long)c.max_batch * c.max_prompt;
    p.teacher_rows = (int)(tr < kTeacherChunk ? tr : kTeacherChunk);
  }
  p.logit_rows = (c.flags & KF_FLAG_DEBUG_LOGITS)
                     ? (p.head_max > p.teacher_rows ? p.head_max : p.teacher_rows)
                     : c.max_batch;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  const size_t es = p.es;
  p.wbegin = off;
  p.tok = take((size_t)p.Vpad * d * es);
  p.pos = take(T * d * es);
  p.nw1 = take(4 * d * d * es);
  p.nb1 = take(4 * d * 4);
  p.nw2 = take(4 * d * d * es);
  p.nb2 = take(d * 4);
  p.omega = take(d / 2 * 8);
  p.layer.resize(L);
  for (size_t l = 0; l < L; ++l) {
    LayerOff& y = p.layer[l];
    y.ln1_g = take(d * 4);
    y.ln1_b = take(d * 4);
    y.wqkv = take(3 * d * d * es);
    y.bqkv = take(3 * d * 4);
    y.wo = take(d * d * es);
    y.bo = take(d * 4);
    y.ln2_g = take(d * 4);
    y.ln2_b = take(d * 4);
    y.w1 = take(f * d * es);
    y.b1 = take(f * 4);
    y.w2 = take(d * f * es);
    y.b2 = take(d * 4);
    y.qkv_c1 = take(3 * d * 4);
    y.qkv_c2 = take(3 * d * 4);
    y.up_c1 = take(f * 4);
    y.up_c2 = take(f * 4);
  }
  p.lnf_g = take(d * 4);
  p.lnf_b = take(d * 4);
  p.head_c1 = take((size_t)p.Vpad * 4);
  p.head_c2 = take((size_t)p.Vpad * 4);
  p.head_w = take((size_t)p.Vpad * d * es);
  if (c.flags & KF_FLAG_RMS_ROPE) p.rope = take(T * 32 * sizeof(float2));
  if (c.flags & KF_FLAG_TEMPERATURE) {
    p.tw1 = take(d * d * es);
    p.tb1 = take(d * 4);
    p.tw2 = take(d * d * es);
    p.tb2 = take(d * 4);
  }
  p.wend = off;
  p.Tp = (c.n_ctx + kPage - 1) / kPage * kPage;
  p.npp = p.Tp / kPage;
  p.page_bytes = L * 2 * d * kPage * es;
  p.n_pages = c.kv_pages > 0 ? c.kv_pages : c.max_batch * p.npp;
  p.kv_bytes = (size_t)p.n_pages * p.page_bytes;
  p.kv = take(p.kv_bytes);
  if (c.flags & KF_FLAG_SERVING) {
    p.meta = take((size_t)c.max_batch * (2 + p.npp) * 4);
    p.serve_noise = take((size_t)c.max_batch * c.max_k * 4);
    p.serve_out = take((size_t)c.max_batch * c.max_k * 4);
  }
  const size_t R = p.rows_max, Hw = f > 4 * d ? f : 4 * d;
  p.X = take(R * d * 4);
  p.temb = (c.flags & KF_FLAG_TEMPERATURE) ? take((size_t)c.max_batch * d * es) : 0;
  p.Xh = es == 2 ? take(R * d * es) : p.X;
  p.lnst = take(R * (d / 16) * 8);  // LayerNorm partial sums of the residual rows
  p.A = take(R * d * es);
  p.Q = take(R * d * es);
  p.O = take(R * d * es);
  p.Hm = take(R * Hw * es);
  p.noise = take((size_t)p.head_max * 4);
  p.pval = take((size_t)p.head_max * p.n_tiles * 4);
  p.pidx = take((size_t)p.head_max * p.n_tiles * 4);
  p.logits = take((size_t)p.logit_rows * c.vocab * 4);
  if (c.flags & KF_FLAG_ROLLOUT)
    p.roll_kv = take(L * 2 * (size_t)c.max_batch * c.n_head *
                     ((size_t)c.max_prompt * (1 + 2 * (size_t)c.max_k)) * (d / c.n_head) * es);
  p.tmax = take((size_t)p.teacher_rows * p.n_tiles * 4);
  p.tsub = take((size_t)p.teacher_rows * p.n_tiles * 8 * 4);
  p.dstate = take(sizeof(KfDevState));
  p.pend = take((size_t)c.max_batch * c.max_k * 4);
  p.att_m = take((size_t)kAttnEntries * 4);
  p.att_l = take((size_t)kAttnEntries * 4);
  p.att_o = take((size_t)kAttnEntries * (d / c.n_head) * 4);
  p.split_part = take(kSplitBytes);
  p.nz_rows = kNoiseAheadRows > c.max_batch * c.max_k ? kNoiseAheadRows : c.max_batch * c.max_k;
  p.nzA = take((size_t)p.nz_rows * d * es);
  p.nzH = take((size_t)p.nz_rows * 4 * d * es);
  p.nz = take((size_t)p.nz_rows * d * 4);
  p.total = off;
}

uint16_t f32_to_bf16_rne(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

}  // namespace

// ------------------------------------------------------------------ context
struct kf_ctx {
  kf_config cfg;
  hipStream_t stream = nullptr;
  Plan plan;
  char* base = nullptr;
  size_t bytes = 0;
  bool weights = false;
  // sequence state (host mirror of the device state)
  bool live = false;
  int B = 0, C = 0, pending = 0;
  int temp_B = 0;  // sequences whose temperature embedding is set (kf_set_temperature)
  // continuous batching (KF_FLAG_SERVING): sequence slots and the page pool
  struct Slot {
    bool live = false;
    int C = 0, pending = 0;
    std::vector<int> pages;  // page ids of positions 0, 128, 256, ...
  };
  std::vector<Slot> slots;
  std::vector<int> free_pages;  // stack of unused page ids
  int serving = 0;              // live slots
  std::vector<int> map_dev;     // the slot map last written to the device
  // captured served steps, by (sequences, pending rows, noise rows); most recent last
  struct ServeGraph {
    int n, nr, k;
    hipGraphExec_t exec;
  };
  std::vector<ServeGraph> sgraphs;
  int last_head_rows = 0;
  bool last_logits = false;
  std::string err;
  // kernel timing: bit c set = bracket launches of class c
  int timing = 0;
  struct Ev {
    hipEvent_t a, b;
    int cls;
  };
  std::vector<Ev> evs;
  size_t ev_used = 0;
  bool ev_open = false;
  // device scratch of kf_decode_block_noalloc on the state buffer's GPU (its
  // address from hipGetSymbolAddress), or null with the reason in scratch_err
  char* scratch = nullptr;
  std::string scratch_err;
  // HIP-graph replay of the fixed-shape decode block of a generation run
  bool graphs = true;
  hipGraphExec_t gexec = nullptr;
  struct GraphKey {
    int B, nr, k, N, L;
    uint64_t seed;
    const void* out;
    bool operator==(const GraphKey& o) const {
      return B == o.B && nr == o.nr && k == o.k && N == o.N && L == o.L && seed == o.seed &&
             out == o.out;
    }
  } gkey{};
};

namespace kf {
thread_local LaunchTimer* launch_timer = nullptr;
}  // namespace kf

namespace {

int fail(kf_ctx* c, int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c) c->err = buf;
  return code;
}

int hip_fail(kf_ctx* c, hipError_t e, const char* what) {
  return fail(c, KF_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define KF_HIP(ctx, expr)                                        \
  do {                                                           \
    hipError_t e_ = (expr);                                      \
    if (e_ != hipSuccess) return hip_fail((ctx), e_, #expr);     \
  } while (0)

// Timing of one launcher call of class cls: its kernels record the event pair
// themselves (kf::launch_timer); a call that launched nothing is dropped.
thread_local kf::LaunchTimer g_timer;

int ev_begin(kf_ctx* c, int cls) {
  c->ev_open = false;
  if (!(c->timing & (1 << cls))) return 0;
  if (c->ev_used == c->evs.size()) {
    kf_ctx::Ev e;
    KF_HIP(c, hipEventCreate(&e.a));
    KF_HIP(c, hipEventCreate(&e.b));
    c->evs.push_back(e);
  }
  kf_ctx::Ev& e = c->evs[c->ev_used];
  e.cls = cls;
  g_timer = kf::LaunchTimer{e.a, e.b, false};
  kf::launch_timer = &g_timer;
  c->ev_open = true;
  return 0;
}

int ev_end(kf_ctx* c) {
  if (!c->ev_open) return 0;
  c->ev_open = false;
  kf::launch_timer = nullptr;
  if (g_timer.started) ++c->ev_used;
  return 0;
}

#define KF_LAUNCH(ctx, cls, expr)                                \
  do {                                                           \
    int r_ = ev_begin((ctx), (cls));                             \
    if (r_) return r_;                                           \
    hipError_t e_ = (expr);                                      \
    ev_end((ctx));                                               \
    if (e_ != hipSuccess) return hip_fail((ctx), e_, #expr);     \
  } while (0)

// Partial-result buffers of one step (attention key-split states, split-K
// parts, head argmax partials).
struct Scratch {
  float *att_m, *att_l, *att_o;
  int att_entries;
  float* split;
  size_t split_bytes;
  float* pval;
  int* pidx;
};

// Inputs of one step.
struct StepIn {
  int B, nr, k;              // sequences, real rows, noise rows (k == 0: AR step)
  const int32_t* toks;       // real-row tokens [B][tok_stride] (or [slots][..], see serve)
  int tok_stride;
  const float* noise;        // [B][k] or null (device Philox)
  const float* u_ar;         // AR: [B] or null (device Philox)
  uint64_t seed;
  KfOutDesc od;
  bool reset;                // prefill: C := 0 before the step
  // teacher targets (kf_teacher_targets): every real row is sampled
  const float* tau = nullptr;    // [B] temperatures
  const float* u_rows = nullptr; // [B][nr] noise
  int32_t* targets = nullptr;    // [B][nr] output; non-null selects the teacher head
  // continuous batching: step sequence b is the slot in the device slot map,
  // with its own committed length and pages; toks are then indexed by slot
  // when toks_by_slot (the pending-token buffer)
  bool serve = false;
  bool toks_by_slot = false;
  // kf_decode_block_noalloc: partial results in the library's device scratch
  // instead of the state buffer's workspace
  const Scratch* scr = nullptr;
  // kf_generate: the noise rows come from the encoder output computed ahead
  // (the embedding kernel writes them; no noise kernels in the step)
  const kf::NoiseAhead* na = nullptr;
};


template <typename T>
int run_step(kf_ctx* c, const StepIn& in) {
  const Plan& p = c->plan;
  char* base = c->base;
  const kf_config& cf = c->cfg;
  const int d = cf.d_model, f = cf.d_mlp, V = cf.vocab;
  hipStream_t s = c->stream;
  KfDevState* st = reinterpret_cast<KfDevState*>(base + p.dstate);
  float* X = reinterpret_cast<float*>(base + p.X);
  T* Xh = reinterpret_cast<T*>(base + p.Xh);  // compute-dtype residual copy (X itself for fp32)
  float2* lnst = reinterpret_cast<float2*>(base + p.lnst);
  const T* temb = (cf.flags & KF_FLAG_TEMPERATURE) ? reinterpret_cast<const T*>(base + p.temb) : nullptr;
  kf::AttnSplit asp{reinterpret_cast<float*>(base + p.att_m),
                    reinterpret_cast<float*>(base + p.att_l),
                    reinterpret_cast<float*>(base + p.att_o), kAttnEntries, 1};
  kf::SplitWs sws{reinterpret_cast<float*>(base + p.split_part), kSplitBytes};
  float* pval = reinterpret_cast<float*>(base + p.pval);
  int* pidx = reinterpret_cast<int*>(base + p.pidx);
  if (in.scr) {
    asp = kf::AttnSplit{in.scr->att_m, in.scr->att_l, in.scr->att_o, in.scr->att_entries, 1};
    sws = kf::SplitWs{in.scr->split, in.scr->split_bytes};
    pval = in.scr->pval;
    pidx = in.scr->pidx;
  }
  T* A = reinterpret_cast<T*>(base + p.A);  // noise sinusoid staging
  T* Q = reinterpret_cast<T*>(base + p.Q);
  T* O = reinterpret_cast<T*>(base + p.O);
  T* Hm = reinterpret_cast<T*>(base + p.Hm);
  T* kv = reinterpret_cast<T*>(base + p.kv);
  const T* tok = reinterpret_cast<const T*>(base + p.tok);
  const T* pos = reinterpret_cast<const T*>(base + p.pos);
  auto F = [&](size_t o) { return reinterpret_cast<const float*>(base + o); };
  auto W = [&](size_t o) { return reinterpret_cast<const T*>(base + o); };

  KfStepGeom g{in.B, in.nr + in.k, in.nr, in.k};
  KfKvGeom kg{cf.n_layer, cf.n_head, p.Tp, d / cf.n_head};
  if (in.serve) {
    int* meta = reinterpret_cast<int*>(base + p.meta);
    g.map = meta;
    g.cs = meta + cf.max_batch;
    kg.ptab = meta + 2 * cf.max_batch;
  }
  const int M = in.B * g.R;
  const bool debug = (cf.flags & KF_FLAG_DEBUG_LOGITS) != 0;
  const int rms = (cf.flags & KF_FLAG_RMS_ROPE) ? 1 : 0;
  const float2* rope = rms ? reinterpret_cast<const float2*>(base + p.rope) : nullptr;

  if (in.reset && in.serve) KF_HIP(c, kf::launch_seq_reset(g, s));
  else if (in.reset) KF_HIP(c, kf::launch_zero_i32(reinterpret_cast<int*>(st), 1, s));
  if (in.nr > 0 || (in.na && in.k > 0))
    KF_LAUNCH(c, KF_KC_EMBED,
              kf::launch_embed_real<T>(X, Xh, lnst, tok, pos, in.toks, in.tok_stride,
                                       in.toks_by_slot ? 1 : 0, g, d, V, st, s,
                                       in.k > 0 ? in.na : nullptr));
  if (in.k > 0 && !in.na) {
    const int Mk = in.B * in.k;
    float* urec = reinterpret_cast<float*>(base + p.noise);
    KF_LAUNCH(c, KF_KC_NOISE,
              kf::launch_noise_sinusoid<T>(A, in.noise, in.seed,
                                           reinterpret_cast<const double*>(base + p.omega), g, d,
                                           st, urec, s));
    KF_LAUNCH(c, KF_KC_NOISE,
              kf::gemm_bias<T>(A, W(p.nw1), Mk, 4 * d, d, F(p.nb1), kf::Act::Gelu, Hm, 4 * d, &sws, s));
    KF_LAUNCH(c, KF_KC_NOISE,
              kf::gemm_noise_out<T>(Hm, W(p.nw2), Mk, d, 4 * d, F(p.nb2), pos, temb, X, Xh, lnst, g,
                                    st, &sws, s));
  }
  // The teacher pass of a 16-bit model (causal attention over whole sequences,
  // nothing decoded after it) runs its attention through the block kernel of
  // the training masks: SingleForward with no noise rows is the causal mask.
  // Q goes to [B][H][N][d_head] and K, V to two such buffers in the KV cache
  // memory, which the pass does not otherwise use.
  const bool seq_attn = in.targets && sizeof(T) == 2;
  const int H = cf.n_head, dh = d / cf.n_head;
  for (int l = 0; l < cf.n_layer; ++l) {
    const LayerOff& y = p.layer[l];
    const kf::LnFold ln1{F(y.qkv_c1), F(y.qkv_c2), lnst, rms};
    const kf::LnFold ln2{F(y.up_c1), F(y.up_c2), lnst, rms};
    if constexpr (sizeof(T) == 2) {
      if (seq_attn) {
        const int n = in.nr;
        T* Kl = kv;
        T* Vl = kv + (size_t)in.B * n * d;
        KF_LAUNCH(c, KF_KC_QKV,
                  kf::gemm_qkv_seq<T>(Xh, ln1, W(y.wqkv), M, d, F(y.bqkv), Q, Kl, Vl, n, n, 0, H,
                                      n, 0, 1, rope, s));
        KF_LAUNCH(c, KF_KC_ATTN,
                  kf::launch_training_attention_seq(KF_MASK_SINGLE, in.B, H, n, 0, dh, Q, Kl, Vl,
                                                    n, O, 1.0f / sqrtf((float)dh), s));
      }
    }
    // In the last layer of a step with noise rows only the noise rows go on
    // past the KV append: the head reads nothing else, and the real rows'
    // K and V are already in the cache (Appendix C.1: only the noise outputs
    // are decoded).  Attention, out-projection and MLP run at M = B k
    // (OWT-shaped batch 512 +0.9 %, the 24-layer backbone +0.5 %).  Steps of
    // at most 16 rows keep all rows: their GEMMs cost one memory round trip
    // whatever the row count (batch 1: -0.6 % with the head rows only).
    const bool head_only =
        l == cf.n_layer - 1 && in.k > 0 && in.nr > 0 && !in.targets && M > 16;
    if (!seq_attn) {
      KF_LAUNCH(c, KF_KC_QKV,
                kf::gemm_qkv_ln<T>(Xh, ln1, W(y.wqkv), M, d, F(y.bqkv), Q, kv, g, kg, l, st, rope, s));
      KfStepGeom ga = g;
      if (head_only) ga.qoff = in.nr;
      KF_LAUNCH(c, KF_KC_ATTN, kf::launch_attention<T>(Q, kv, O, st, ga, kg, l, asp, s));
    }
    if (head_only) {
      const int Mh = in.B * in.k;
      KF_LAUNCH(c, KF_KC_OPROJ,
                kf::gemm_residual_rows<T>(O, true, g, W(y.wo), Mh, d, d, F(y.bo), X, Xh, lnst, &sws, s));
      KF_LAUNCH(c, KF_KC_MLP_UP,
                kf::gemm_up_ln_rows<T>(Xh, ln2, g, W(y.w1), Mh, f, d, F(y.b1), Hm, s));
      KF_LAUNCH(c, KF_KC_MLP_DOWN,
                kf::gemm_residual_rows<T>(Hm, false, g, W(y.w2), Mh, d, f, F(y.b2), X, Xh, lnst, &sws,
                                          s));
      continue;
    }
    KF_LAUNCH(c, KF_KC_OPROJ, kf::gemm_residual<T>(O, W(y.wo), M, d, d, F(y.bo), X, Xh, lnst, &sws, s));
    KF_LAUNCH(c, KF_KC_MLP_UP, kf::gemm_up_ln<T>(Xh, ln2, W(y.w1), M, f, d, F(y.b1), Hm, s));
    KF_LAUNCH(c, KF_KC_MLP_DOWN, kf::gemm_residual<T>(Hm, W(y.w2), M, d, f, F(y.b2), X, Xh, lnst, &sws, s));
  }
  if (in.targets) {
    // Teacher targets: the sampling head over every row, in chunks of the
    // head-partials workspace, each followed by its inverse-CDF selection.
    const kf::LnFold lnf{F(p.head_c1), F(p.head_c2), lnst, rms};
    float* tmax = reinterpret_cast<float*>(base + p.tmax);
    float* tsub = reinterpret_cast<float*>(base + p.tsub);
    float* lg = debug ? reinterpret_cast<float*>(base + p.logits) : nullptr;
    int mc = 0;
    for (int r0 = 0; r0 < M; r0 += p.teacher_rows) {
      mc = M - r0 < p.teacher_rows ? M - r0 : p.teacher_rows;
      KF_LAUNCH(c, KF_KC_HEAD,
                kf::gemm_head_sample<T>(Xh, lnf, W(p.head_w), mc, p.Vpad, V, d, r0, in.nr, in.tau,
                                        tmax, tsub, lg, s));
      KF_LAUNCH(c, KF_KC_SELECT,
                kf::launch_teacher_select<T>(tmax, tsub, p.n_tiles, V, Xh, lnst, W(p.head_w),
                                             F(p.head_c1), F(p.head_c2), rms, d, in.tau, in.u_rows,
                                             r0, mc, in.nr, in.targets, st, s));
    }
    c->last_head_rows = mc;
    c->last_logits = debug;
    return KF_OK;
  }
  const bool ar = in.k == 0;
  const int Mh = ar ? in.B : in.B * in.k;
  float* logits = (ar || debug) ? reinterpret_cast<float*>(base + p.logits) : nullptr;
  const kf::LnFold lnf{F(p.head_c1), F(p.head_c2), lnst, rms};
  // The argmax head commits the step itself (its first workgroup, C += nr),
  // which saves the commit launch; the AR path commits after its sampler.
  KF_LAUNCH(c, KF_KC_HEAD,
            kf::gemm_head_ln<T>(Xh, lnf, W(p.head_w), Mh, p.Vpad, V, d, ar ? 2 : 1, g, pval, pidx,
                                logits, s, ar ? nullptr : st, in.nr));
  if (!ar) {
    KF_LAUNCH(c, KF_KC_SELECT,
              kf::launch_argmax_select(pval, pidx, p.n_tiles, g, st, in.od, s, in.nr));
  } else {
    KF_LAUNCH(c, KF_KC_SELECT,
              kf::launch_icdf_select(logits, V, in.u_ar, in.seed, g, st, in.od, s));
    KF_LAUNCH(c, KF_KC_SELECT, kf::launch_commit(st, g, in.nr, s));
  }
  c->last_head_rows = Mh;
  c->last_logits = logits != nullptr;
  return KF_OK;
}

// Stage-2 self-forcing teacher rollout (Appendix C.2): round 1 is a
// SingleForward pass over [context N | noise N*k] rows per sequence, its
// noise rows' argmax giving x1; round 2 a DoubleForward pass over
// [Future-1 N*k | Future-2 N*k] rows (x1 as tokens, then fresh noise) that
// attends to round 1's context keys, its Future-2 argmax giving x2.  Each
// layer's keys and values live in one buffer [B][H][N + 2Nk][dh]:
// [context | noise of round 1, then Future-1 | Future-2].
template <typename T>
int run_rollout(kf_ctx* c, int B, int N, int k, const int32_t* tokens, const float* z1,
                const float* z2, int32_t* x1, int32_t* x2) {
  const Plan& p = c->plan;
  char* base = c->base;
  const kf_config& cf = c->cfg;
  const int d = cf.d_model, f = cf.d_mlp, V = cf.vocab, H = cf.n_head, dh = d / H;
  hipStream_t s = c->stream;
  KfDevState* st = reinterpret_cast<KfDevState*>(base + p.dstate);
  float* X = reinterpret_cast<float*>(base + p.X);
  T* Xh = reinterpret_cast<T*>(base + p.Xh);
  float2* lnst = reinterpret_cast<float2*>(base + p.lnst);
  const T* temb = (cf.flags & KF_FLAG_TEMPERATURE) ? reinterpret_cast<const T*>(base + p.temb) : nullptr;
  const kf::SplitWs sws{reinterpret_cast<float*>(base + p.split_part), kSplitBytes};
  T* A = reinterpret_cast<T*>(base + p.A);
  T* Q = reinterpret_cast<T*>(base + p.Q);
  T* O = reinterpret_cast<T*>(base + p.O);
  T* Hm = reinterpret_cast<T*>(base + p.Hm);
  const T* tok = reinterpret_cast<const T*>(base + p.tok);
  const T* pos = reinterpret_cast<const T*>(base + p.pos);
  auto F = [&](size_t o) { return reinterpret_cast<const float*>(base + o); };
  auto W = [&](size_t o) { return reinterpret_cast<const T*>(base + o); };
  const int ldk = N * (1 + 2 * k), nk = N * k;
  const size_t kvl = (size_t)B * H * ldk * dh;  // elements of one layer's K (or V)
  T* kvb = reinterpret_cast<T*>(base + p.roll_kv);
  const bool debug = (cf.flags & KF_FLAG_DEBUG_LOGITS) != 0;
  float* logits = debug ? reinterpret_cast<float*>(base + p.logits) : nullptr;
  const int rms = (cf.flags & KF_FLAG_RMS_ROPE) ? 1 : 0;
  const float2* rope = rms ? reinterpret_cast<const float2*>(base + p.rope) : nullptr;

  auto noise = [&](const float* z, int n, int off, int shift) -> int {
    const KfStepGeom gz{B * N, k, 0, k};  // one noise group of k per (sequence, position)
    KF_LAUNCH(c, KF_KC_NOISE,
              kf::launch_noise_sinusoid<T>(A, z, 0, reinterpret_cast<const double*>(base + p.omega),
                                           gz, d, st, nullptr, s));
    KF_LAUNCH(c, KF_KC_NOISE,
              kf::gemm_bias<T>(A, W(p.nw1), B * nk, 4 * d, d, F(p.nb1), kf::Act::Gelu, Hm, 4 * d,
                               &sws, s));
    KF_LAUNCH(c, KF_KC_NOISE,
              kf::gemm_seq_noise_out<T>(Hm, W(p.nw2), B * nk, d, 4 * d, F(p.nb2), pos, temb, X, Xh,
                                        lnst, n, off, N, k, shift, &sws, s));
    return KF_OK;
  };
  auto body = [&](int n, int koff, int mask) -> int {
    const int M = B * n;
    const int round = mask == KF_MASK_SINGLE ? 1 : 2;
    for (int l = 0; l < cf.n_layer; ++l) {
      const LayerOff& y = p.layer[l];
      const kf::LnFold ln1{F(y.qkv_c1), F(y.qkv_c2), lnst, rms};
      const kf::LnFold ln2{F(y.up_c1), F(y.up_c2), lnst, rms};
      T* Kl = kvb + (size_t)l * 2 * kvl;
      T* Vl = Kl + kvl;
      KF_LAUNCH(c, KF_KC_QKV,
                kf::gemm_qkv_seq<T>(Xh, ln1, W(y.wqkv), M, d, F(y.bqkv), Q, Kl, Vl, n, ldk, koff, H,
                                    N, k, round, rope, s));
      KF_LAUNCH(c, KF_KC_ATTN,
                kf::launch_training_attention_seq(mask, B, H, N, k, dh, reinterpret_cast<const bf16*>(Q),
                                                  reinterpret_cast<const bf16*>(Kl),
                                                  reinterpret_cast<const bf16*>(Vl), ldk,
                                                  reinterpret_cast<bf16*>(O), 1.0f / sqrtf((float)dh), s));
      KF_LAUNCH(c, KF_KC_OPROJ, kf::gemm_residual<T>(O, W(y.wo), M, d, d, F(y.bo), X, Xh, lnst, &sws, s));
      KF_LAUNCH(c, KF_KC_MLP_UP, kf::gemm_up_ln<T>(Xh, ln2, W(y.w1), M, f, d, F(y.b1), Hm, s));
      KF_LAUNCH(c, KF_KC_MLP_DOWN,
                kf::gemm_residual<T>(Hm, W(y.w2), M, d, f, F(y.b2), X, Xh, lnst, &sws, s));
    }
    return KF_OK;
  };
  auto head = [&](int n, int off, int32_t* out) -> int {
    const KfStepGeom gh{B, n, off, nk};  // head rows: the nk rows after `off` of each sequence
    const kf::LnFold lnf{F(p.head_c1), F(p.head_c2), lnst, rms};
    KF_LAUNCH(c, KF_KC_HEAD,
              kf::gemm_head_ln<T>(Xh, lnf, W(p.head_w), B * nk, p.Vpad, V, d, 1, gh,
                                  reinterpret_cast<float*>(base + p.pval),
                                  reinterpret_cast<int*>(base + p.pidx), logits, s));
    KfOutDesc od;
    od.out = out;
    od.stride = nk;
    od.gen_base = -1;
    od.pend = nullptr;
    od.pend_stride = 0;
    KF_LAUNCH(c, KF_KC_SELECT,
              kf::launch_argmax_select(reinterpret_cast<const float*>(base + p.pval),
                                       reinterpret_cast<const int*>(base + p.pidx), p.n_tiles, gh,
                                       st, od, s));
    return KF_OK;
  };

  KF_HIP(c, kf::launch_zero_i32(reinterpret_cast<int*>(st), 1, s));  // C = 0: context positions 0..N-1
  // round 1: SingleForward over [context | noise z1]
  const int n1 = N + nk;
  KF_LAUNCH(c, KF_KC_EMBED,
            kf::launch_embed_real<T>(X, Xh, lnst, tok, pos, tokens, N, 0, KfStepGeom{B, n1, N, 0}, d, V,
                                     st, s));
  if (int r = noise(z1, n1, N, 1)) return r;
  if (int r = body(n1, 0, KF_MASK_SINGLE)) return r;
  if (int r = head(n1, N, x1)) return r;
  // round 2: DoubleForward over [Future-1 = x1 | Future-2 = noise z2]
  const int n2 = 2 * nk;
  KF_LAUNCH(c, KF_KC_EMBED,
            kf::launch_embed_group<T>(X, Xh, lnst, tok, pos, x1, B, N, k, n2, 0, 1, d, V, st, s));
  if (int r = noise(z2, n2, nk, 1 + k)) return r;
  if (int r = body(n2, N, KF_MASK_DOUBLE)) return r;
  if (int r = head(n2, nk, x2)) return r;
  c->last_head_rows = B * nk;
  c->last_logits = debug;
  return KF_OK;
}

int step(kf_ctx* c, const StepIn& in) {
  return c->cfg.dtype == KF_BF16 ? run_step<bf16>(c, in) : run_step<float>(c, in);
}

int ready(kf_ctx* c) {
  if (!c->base) return fail(c, KF_ESTATE, "no state buffer bound (kf_bind_state)");
  if (!c->weights) return fail(c, KF_ESTATE, "no weights loaded (kf_load_weights)");
  return KF_OK;
}

// A temperature-conditioned model embeds noise rows only for sequences whose
// temperature has been set.
int temp_ready(kf_ctx* c, int B) {
  if ((c->cfg.flags & KF_FLAG_TEMPERATURE) && c->temp_B < B)
    return fail(c, KF_ESTATE, "temperature set for %d sequences, the step has %d (kf_set_temperature)",
                c->temp_B, B);
  return KF_OK;
}

KfOutDesc out_desc(kf_ctx* c, int32_t* out, int stride, int gen_base) {
  KfOutDesc od;
  od.out = out;
  od.stride = stride;
  od.gen_base = gen_base;
  od.pend = reinterpret_cast<int32_t*>(c->base + c->plan.pend);
  od.pend_stride = c->cfg.max_k;
  return od;
}

int32_t* pend_ptr(kf_ctx* c) { return reinterpret_cast<int32_t*>(c->base + c->plan.pend); }

// Fold each LayerNorm into the GEMM after it: the QKV and MLP-up weights are
// scaled by the gain in place, the head gets a gain-scaled copy of the token
// table (the table itself stays the embedding), and the per-column sums c1, c2
// are computed.  The fold is exact up to the rounding of the scaled weights.
template <typename T>
int fold_layernorms(kf_ctx* c) {
  const Plan& p = c->plan;
  char* base = c->base;
  const int d = c->cfg.d_model, f = c->cfg.d_mlp;
  auto F = [&](size_t o) { return reinterpret_cast<float*>(base + o); };
  auto W = [&](size_t o) { return reinterpret_cast<T*>(base + o); };
  for (const LayerOff& y : p.layer) {
    KF_HIP(c, kf::launch_ln_fold<T>(W(y.wqkv), W(y.wqkv), F(y.ln1_g), F(y.ln1_b), 3 * d, d,
                                    F(y.qkv_c1), F(y.qkv_c2), c->stream));
    KF_HIP(c, kf::launch_ln_fold<T>(W(y.w1), W(y.w1), F(y.ln2_g), F(y.ln2_b), f, d, F(y.up_c1),
                                    F(y.up_c2), c->stream));
  }
  KF_HIP(c, kf::launch_ln_fold<T>(W(p.tok), W(p.head_w), F(p.lnf_g), F(p.lnf_b), p.Vpad, d,
                                  F(p.head_c1), F(p.head_c2), c->stream));
  return KF_OK;
}

void drop_graph(kf_ctx* c) {
  if (c->gexec) (void)hipGraphExecDestroy(c->gexec);
  c->gexec = nullptr;
}

void drop_serve_graphs(kf_ctx* c) {
  for (auto& g : c->sgraphs) (void)hipGraphExecDestroy(g.exec);
  c->sgraphs.clear();
}

// The noise encoder for passes pass0 .. pass0 + npass - 1 of a lock-step
// generate of B sequences (prompt N, k noise rows a pass), into the plan's
// ahead buffers: sinusoids, Linear(d, 4d) + GELU, Linear(4d, d) in fp32
// without its bias (the embedding kernel adds the bias, the position and the
// temperature embedding when the pass runs).  Three launches for the whole
// chunk instead of three in every pass.
template <typename T>
int run_noise_ahead(kf_ctx* c, int B, int k, int N, uint64_t seed, int pass0, int npass) {
  const Plan& p = c->plan;
  char* base = c->base;
  const int d = c->cfg.d_model, M = npass * B * k;
  hipStream_t s = c->stream;
  T* A = reinterpret_cast<T*>(base + p.nzA);
  T* H = reinterpret_cast<T*>(base + p.nzH);
  auto F = [&](size_t o) { return reinterpret_cast<const float*>(base + o); };
  auto W = [&](size_t o) { return reinterpret_cast<const T*>(base + o); };
  KF_LAUNCH(c, KF_KC_NOISE,
            kf::launch_noise_sinusoid_ahead<T>(A, seed, reinterpret_cast<const double*>(base + p.omega),
                                               B, k, N, pass0, npass, d, s));
  KF_LAUNCH(c, KF_KC_NOISE,
            kf::gemm_bias<T>(A, W(p.nw1), M, 4 * d, d, F(p.nb1), kf::Act::Gelu, H, 4 * d, nullptr, s));
  KF_LAUNCH(c, KF_KC_NOISE,
            kf::gemm_f32<T>(H, W(p.nw2), M, d, 4 * d, reinterpret_cast<float*>(base + p.nz), s));
  return KF_OK;
}

int noise_ahead(kf_ctx* c, int B, int k, int N, uint64_t seed, int pass0, int npass) {
  return c->cfg.dtype == KF_BF16 ? run_noise_ahead<bf16>(c, B, k, N, seed, pass0, npass)
                                 : run_noise_ahead<float>(c, B, k, N, seed, pass0, npass);
}

// Run `count` identical steps and advance the host view of C by `adv` after
// each.  Every launch of such a step reads C from device memory, so one
// captured step replays unchanged; the instantiated graph is cached on the
// context for the next call with the same arguments.  Graphs need a real
// stream (capture is impossible on the legacy null stream) and are not used
// while kernel timing is on.
// before(i) runs on the host before decode pass i = 1 .. count is issued
// (between graph replays: it may launch work of its own on the stream).
int repeat_step(kf_ctx* c, const StepIn& in, int count, int adv, int N, int L,
                const std::function<int(int)>& before = nullptr) {
  if (count <= 0) return KF_OK;
  if (!c->graphs || c->stream == nullptr || c->timing) {
    for (int i = 0; i < count; ++i) {
      int r = before ? before(i + 1) : KF_OK;
      if (r) return r;
      r = step(c, in);
      if (r) return r;
      c->C += adv;
    }
    return KF_OK;
  }
  kf_ctx::GraphKey key{in.B, in.nr, in.k, N, L, in.seed, in.od.out};
  if (!c->gexec || !(key == c->gkey)) {
    drop_graph(c);
    KF_HIP(c, hipStreamBeginCapture(c->stream, hipStreamCaptureModeRelaxed));
    int r = step(c, in);
    hipGraph_t g = nullptr;
    hipError_t e = hipStreamEndCapture(c->stream, &g);
    if (r) {
      if (e == hipSuccess && g) (void)hipGraphDestroy(g);
      return r;
    }
    if (e != hipSuccess) return hip_fail(c, e, "hipStreamEndCapture");
    e = hipGraphInstantiate(&c->gexec, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (e != hipSuccess) {
      c->gexec = nullptr;
      return hip_fail(c, e, "hipGraphInstantiate");
    }
    c->gkey = key;
  }
  for (int i = 0; i < count; ++i) {
    if (before) {
      int r = before(i + 1);
      if (r) return r;
    }
    KF_HIP(c, hipGraphLaunch(c->gexec, c->stream));
    c->C += adv;
  }
  return KF_OK;
}

// Temperature embeddings of sequences 0..B-1: tau through the noise sinusoid,
// then Linear(d, d), GELU, Linear(d, d), into temb [b][d].
template <typename T>
int run_temperature(kf_ctx* c, const float* tau, int B) {
  const Plan& p = c->plan;
  char* base = c->base;
  const int d = c->cfg.d_model;
  hipStream_t s = c->stream;
  T* A = reinterpret_cast<T*>(base + p.A);
  T* Hm = reinterpret_cast<T*>(base + p.Hm);
  T* temb = reinterpret_cast<T*>(base + p.temb);
  auto F = [&](size_t o) { return reinterpret_cast<const float*>(base + o); };
  auto W = [&](size_t o) { return reinterpret_cast<const T*>(base + o); };
  const KfStepGeom g{B, 1, 0, 1};  // one "noise row" per sequence, u = tau[b]
  KF_HIP(c, kf::launch_noise_sinusoid<T>(A, tau, 0, reinterpret_cast<const double*>(base + p.omega), g,
                                         d, reinterpret_cast<const KfDevState*>(base + p.dstate),
                                         nullptr, s));
  KF_HIP(c, kf::gemm_bias<T>(A, W(p.tw1), B, d, d, F(p.tb1), kf::Act::Gelu, Hm, d, nullptr, s));
  KF_HIP(c, kf::gemm_bias<T>(Hm, W(p.tw2), B, d, d, F(p.tb2), kf::Act::None, temb, d, nullptr, s));
  return KF_OK;
}

// ------------------------------------------------------ continuous batching
// Host side of the paged KV pool: a stack of free page ids and, per sequence
// slot, the pages that hold its positions 0, 128, 256, ...  The device copy of
// the page table and of the step's slot map is kept current through scatter
// launches (the values travel in the launch arguments).

void serve_reset(kf_ctx* c) {
  c->slots.assign(c->cfg.max_batch, kf_ctx::Slot{});
  c->free_pages.resize(c->plan.n_pages);
  for (int i = 0; i < c->plan.n_pages; ++i) c->free_pages[i] = c->plan.n_pages - 1 - i;
  c->serving = 0;
  c->map_dev.clear();
}

// Lock-step calls address sequence b's pages b * npp + j directly: they end
// every served sequence, and need B whole sequences' worth of pages.
int lockstep_begin(kf_ctx* c, int B) {
  if ((long long)B * c->plan.npp > c->plan.n_pages)
    return fail(c, KF_EINVAL, "B=%d sequences of %d pages exceed the KV pool of %d pages", B,
                c->plan.npp, c->plan.n_pages);
  if (c->serving) serve_reset(c);
  return KF_OK;
}

struct ScatterBatch {
  kf_ctx* c;
  int* dst;
  kf::KfScatter u{};
  int add(int idx, int val) {
    u.idx[u.n] = idx;
    u.val[u.n] = val;
    if (++u.n == kf::kScatterMax) return flush();
    return KF_OK;
  }
  int flush() {
    if (u.n == 0) return KF_OK;
    KF_HIP(c, kf::launch_scatter_i32(dst, u, c->stream));
    u.n = 0;
    return KF_OK;
  }
};

// Check the slot list of a serving call: distinct ids in [0, max_batch).
int check_slots(kf_ctx* c, int n, const int32_t* slots) {
  if (n < 1 || n > c->cfg.max_batch)
    return fail(c, KF_EINVAL, "n=%d outside [1, %d]", n, c->cfg.max_batch);
  if (!slots) return fail(c, KF_EINVAL, "null slot list");
  std::vector<char> seen(c->cfg.max_batch, 0);
  for (int b = 0; b < n; ++b) {
    const int q = slots[b];
    if (q < 0 || q >= c->cfg.max_batch) return fail(c, KF_EINVAL, "slot %d outside [0, %d)", q, c->cfg.max_batch);
    if (seen[q]) return fail(c, KF_EINVAL, "slot %d appears twice", q);
    seen[q] = 1;
  }
  return KF_OK;
}

// Give each slot of the step the pages that cover positions [0, upto[b]),
// all or nothing, and send the new page-table entries and the slot map to the
// device.  On failure nothing changes.
int serve_prepare(kf_ctx* c, int n, const int32_t* slots, const std::vector<int>& upto) {
  const Plan& p = c->plan;
  int need = 0;
  for (int b = 0; b < n; ++b) {
    const int want = (upto[b] + kPage - 1) / kPage;
    const int have = (int)c->slots[slots[b]].pages.size();
    if (want > have) need += want - have;
  }
  if (need > (int)c->free_pages.size())
    return fail(c, KF_ENOMEM, "the step needs %d more KV pages, %zu of %d are free", need,
                c->free_pages.size(), p.n_pages);
  ScatterBatch sb{c, reinterpret_cast<int*>(c->base + p.meta)};
  for (int b = 0; b < n; ++b) {
    kf_ctx::Slot& sl = c->slots[slots[b]];
    const int want = (upto[b] + kPage - 1) / kPage;
    while ((int)sl.pages.size() < want) {
      const int pg = c->free_pages.back();
      c->free_pages.pop_back();
      const int j = (int)sl.pages.size();
      sl.pages.push_back(pg);
      if (int r = sb.add(2 * c->cfg.max_batch + slots[b] * p.npp + j, pg)) return r;
    }
  }
  if ((int)c->map_dev.size() < n) c->map_dev.resize(n, -1);
  for (int b = 0; b < n; ++b)
    if (c->map_dev[b] != slots[b]) {
      if (int r = sb.add(b, slots[b])) return r;
      c->map_dev[b] = slots[b];
    }
  return sb.flush();
}

void serve_free(kf_ctx* c, int q) {
  kf_ctx::Slot& sl = c->slots[q];
  for (int pg : sl.pages) c->free_pages.push_back(pg);
  sl = kf_ctx::Slot{};
  --c->serving;
}

}  // namespace

// ==================================================================== ABI
extern "C" {

// ------------------------------------------------ decode without allocation
// The partial results of kf_decode_block_noalloc live in this file-scope
// device array, one copy per GPU the library runs on, kept until the process
// ends.  In host code its name is not a device address: each GPU's copy is
// found once through hipGetSymbolAddress with that GPU current, and only that
// address is used afterwards.  Regions (256-byte aligned): attention key-split
// states m, l [entries] and o [entries][128]; split-K parts; head argmax
// values and indices [entries] each.
namespace {
constexpr size_t kNaAttnM = 0;
constexpr size_t kNaAttnL = kNaAttnM + (size_t)KF_NOALLOC_ATTN_ENTRIES * 4;
constexpr size_t kNaAttnO = kNaAttnL + (size_t)KF_NOALLOC_ATTN_ENTRIES * 4;
constexpr size_t kNaSplit = kNaAttnO + (size_t)KF_NOALLOC_ATTN_ENTRIES * 128 * 4;
constexpr size_t kNaPval = kNaSplit + (size_t)KF_NOALLOC_SPLIT_BYTES;
constexpr size_t kNaPidx = kNaPval + (size_t)KF_NOALLOC_HEAD_ENTRIES * 4;
constexpr size_t kNaEnd = kNaPidx + (size_t)KF_NOALLOC_HEAD_ENTRIES * 4;
static_assert(kNaEnd == KF_NOALLOC_SCRATCH_BYTES, "scratch layout");
static_assert(kNaAttnL % 256 == 0 && kNaAttnO % 256 == 0 && kNaSplit % 256 == 0 &&
                  kNaPval % 256 == 0 && kNaPidx % 256 == 0,
              "aligned regions");
}  // namespace

static __device__ __align__(256) char scratch[KF_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch[kMaxDevices] = {};

// Address of the scratch copy on the GPU that holds ctx's state buffer,
// looked up once per GPU (with that GPU current).  A failure is kept in
// scratch_err and reported by kf_decode_block_noalloc only.
void find_scratch(kf_ctx* c) {
  c->scratch = nullptr;
  c->scratch_err.clear();
  hipPointerAttribute_t at{};
  hipError_t e = hipPointerGetAttributes(&at, c->base);
  if (e != hipSuccess) {
    c->scratch_err = std::string("hipPointerGetAttributes: ") + hipGetErrorString(e);
    (void)hipGetLastError();  // not left for the launch checks of later calls
    return;
  }
  const int dev = at.device;
  if (dev < 0 || dev >= kMaxDevices) {
    c->scratch_err = "state buffer on device " + std::to_string(dev) + ", beyond the scratch table";
    return;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    int cur = -1;
    e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
    void* ptr = nullptr;
    if (e == hipSuccess) e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (cur >= 0 && cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !ptr) {
      c->scratch_err = std::string("hipGetSymbolAddress(scratch): ") +
                       (e != hipSuccess ? hipGetErrorString(e) : "null address");
      (void)hipGetLastError();
      return;
    }
    g_scratch[dev] = static_cast<char*>(ptr);
  }
  c->scratch = g_scratch[dev];
}
}  // namespace

const char* kf_strerror(int code) {
  switch (code) {
    case KF_OK: return "ok";
    case KF_EINVAL: return "invalid argument";
    case KF_ESTATE: return "invalid state";
    case KF_ECTX: return "context length exceeded";
    case KF_ENOMEM: return "out of memory (state buffer or KV page pool)";
    case KF_EHIP: return "HIP runtime error";
    default: return "unknown error";
  }
}

const char* kf_last_error(const kf_ctx* c) { return c ? c->err.c_str() : "null context"; }

size_t kf_state_bytes(const kf_config* cfg) {
  if (!cfg || !config_ok(*cfg, nullptr)) return 0;
  Plan p;
  make_plan(*cfg, p);
  return p.total;
}

int kf_create(const kf_config* cfg, void* hip_stream, kf_ctx** out) {
  if (!cfg || !out) return KF_EINVAL;
  std::string why;
  if (!config_ok(*cfg, &why)) return KF_EINVAL;
  kf_ctx* c = new (std::nothrow) kf_ctx();
  if (!c) return KF_ENOMEM;
  c->cfg = *cfg;
  c->stream = reinterpret_cast<hipStream_t>(hip_stream);
  make_plan(*cfg, c->plan);
  *out = c;
  return KF_OK;
}

void kf_destroy(kf_ctx* c) {
  if (!c) return;
  drop_graph(c);
  drop_serve_graphs(c);
  for (auto& e : c->evs) {
    (void)hipEventDestroy(e.a);
    (void)hipEventDestroy(e.b);
  }
  delete c;
}

int kf_bind_state(kf_ctx* c, void* dev_ptr, size_t bytes) {
  if (!c) return KF_EINVAL;
  if (!dev_ptr) return fail(c, KF_EINVAL, "null state pointer");
  if (reinterpret_cast<uintptr_t>(dev_ptr) & 255) return fail(c, KF_EINVAL, "state pointer must be 256-byte aligned");
  if (bytes < c->plan.total)
    return fail(c, KF_ENOMEM, "state buffer has %zu bytes, %zu needed", bytes, c->plan.total);
  drop_graph(c);
  drop_serve_graphs(c);
  c->base = static_cast<char*>(dev_ptr);
  c->bytes = bytes;
  c->weights = false;
  c->live = false;
  c->B = c->C = c->pending = 0;
  serve_reset(c);
  find_scratch(c);
  return KF_OK;
}

int kf_load_weights(kf_ctx* c, const void* blob, size_t bytes, int blob_is_device) {
  if (!c) return KF_EINVAL;
  if (!c->base) return fail(c, KF_ESTATE, "no state buffer bound (kf_bind_state)");
  if (!blob) return fail(c, KF_EINVAL, "null blob");
  if (blob_is_device != 0 && blob_is_device != 1) return fail(c, KF_EINVAL, "blob_is_device must be 0 or 1");
  const kf_config& cf = c->cfg;
  const Plan& p = c->plan;
  drop_graph(c);
  const size_t d = cf.d_model, f = cf.d_mlp, V = cf.vocab, T = cf.n_ctx, L = cf.n_layer;
  const bool temp = (cf.flags & KF_FLAG_TEMPERATURE) != 0;
  const bool rmsr = (cf.flags & KF_FLAG_RMS_ROPE) != 0;
  const size_t n_params = V * d + T * d + 8 * d * d + 4 * d + d +
                          L * (2 * d + 3 * d * d + 3 * d + d * d + d + 2 * d + f * d + f + d * f + d) +
                          2 * d + (temp ? 2 * d * d + 2 * d : 0);
  if (bytes != (kHeaderInts + n_params) * 4)
    return fail(c, KF_EINVAL, "blob has %zu bytes, %zu expected for this config", bytes,
                (kHeaderInts + n_params) * 4);
  int32_t hdr[kHeaderInts];
  if (blob_is_device)
    KF_HIP(c, hipMemcpy(hdr, blob, sizeof hdr, hipMemcpyDeviceToHost));
  else
    memcpy(hdr, blob, sizeof hdr);
  const int32_t want[10] = {kMagic, 1, cf.n_layer, cf.d_model, cf.n_head, cf.d_mlp, cf.vocab,
                            cf.n_ctx, cf.dtype,
                            (temp ? kBlobTemperature : 0) | (rmsr ? kBlobRmsRope : 0)};
  for (int i = 0; i < 10; ++i)
    if (hdr[i] != want[i]) return fail(c, KF_EINVAL, "blob header word %d is %d, expected %d", i, hdr[i], want[i]);

  // Destination of each tensor in blob order: (offset, count, is_matrix,
  // unused).  The rotary RMSNorm backbone has no learned positions and no
  // norm shifts: those tensors are skipped and their regions hold zeros.
  struct Dst { size_t off, n; bool mat, unused; };
  std::vector<Dst> dst;
  dst.push_back({p.tok, V * d, true, false});
  dst.push_back({p.pos, T * d, true, rmsr});
  dst.push_back({p.nw1, 4 * d * d, true});
  dst.push_back({p.nb1, 4 * d, false});
  dst.push_back({p.nw2, 4 * d * d, true});
  dst.push_back({p.nb2, d, false});
  for (size_t l = 0; l < L; ++l) {
    const LayerOff& y = p.layer[l];
    dst.push_back({y.ln1_g, d, false});
    dst.push_back({y.ln1_b, d, false, rmsr});
    dst.push_back({y.wqkv, 3 * d * d, true});
    dst.push_back({y.bqkv, 3 * d, false});
    dst.push_back({y.wo, d * d, true});
    dst.push_back({y.bo, d, false});
    dst.push_back({y.ln2_g, d, false});
    dst.push_back({y.ln2_b, d, false, rmsr});
    dst.push_back({y.w1, f * d, true});
    dst.push_back({y.b1, f, false});
    dst.push_back({y.w2, d * f, true});
    dst.push_back({y.b2, d, false});
  }
  dst.push_back({p.lnf_g, d, false});
  dst.push_back({p.lnf_b, d, false, rmsr});
  if (temp) {
    dst.push_back({p.tw1, d * d, true});
    dst.push_back({p.tb1, d, false});
    dst.push_back({p.tw2, d * d, true});
    dst.push_back({p.tb2, d, false});
  }

  // sinusoid frequencies omega_i = 10000^(-i/(d/2)) for the noise encoder
  std::vector<double> omega(d / 2);
  for (size_t i = 0; i < d / 2; ++i) omega[i] = pow(10000.0, -(double)i / (double)(d / 2));
  // rotary table: position p, pair i < d_rot/2 -> (cos, sin) of p 10000^(-2i/d_rot)
  std::vector<float2> rope_cs;
  if (rmsr) {
    const int dh = cf.d_model / cf.n_head, dr = dh < 64 ? dh : 64;
    rope_cs.assign(T * 32, make_float2(0.f, 0.f));
    for (size_t q = 0; q < T; ++q)
      for (int i = 0; i < dr / 2; ++i) {
        const double a = (double)q * pow(10000.0, -2.0 * i / (double)dr);
        rope_cs[q * (dr / 2) + i] = make_float2((float)cos(a), (float)sin(a));
      }
  }

  const bool bf = cf.dtype == KF_BF16;
  if (!blob_is_device) {
    std::vector<uint8_t> img(p.wend - p.wbegin, 0);
    const float* src = static_cast<const float*>(blob) + kHeaderInts;
    for (const Dst& t : dst) {
      uint8_t* o = img.data() + (t.off - p.wbegin);
      if (t.unused) {  // stays zero
      } else if (t.mat && bf) {
        uint16_t* h = reinterpret_cast<uint16_t*>(o);
        for (size_t i = 0; i < t.n; ++i) h[i] = f32_to_bf16_rne(src[i]);
      } else {
        memcpy(o, src, t.n * 4);
      }
      src += t.n;
    }
    memcpy(img.data() + (p.omega - p.wbegin), omega.data(), omega.size() * 8);
    if (rmsr) memcpy(img.data() + (p.rope - p.wbegin), rope_cs.data(), rope_cs.size() * sizeof(float2));
    KF_HIP(c, hipMemcpyAsync(c->base + p.wbegin, img.data(), img.size(), hipMemcpyHostToDevice, c->stream));
    KF_HIP(c, hipStreamSynchronize(c->stream));
  } else {
    const float* src = static_cast<const float*>(blob) + kHeaderInts;
    // padding rows of the head / token table stay zero
    const size_t pad = ((size_t)p.Vpad - V) * d;
    if (bf) {
      KF_HIP(c, kf::launch_zero<bf16>(reinterpret_cast<bf16*>(c->base + p.tok) + V * d, pad, c->stream));
    } else {
      KF_HIP(c, kf::launch_zero<float>(reinterpret_cast<float*>(c->base + p.tok) + V * d, pad, c->stream));
    }
    for (const Dst& t : dst) {
      if (t.unused && t.mat && bf)
        KF_HIP(c, kf::launch_zero<bf16>(reinterpret_cast<bf16*>(c->base + t.off), t.n, c->stream));
      else if (t.unused && t.mat)
        KF_HIP(c, kf::launch_zero<float>(reinterpret_cast<float*>(c->base + t.off), t.n, c->stream));
      else if (t.unused)
        KF_HIP(c, kf::launch_zero<float>(reinterpret_cast<float*>(c->base + t.off), t.n, c->stream));
      else if (t.mat && bf)
        KF_HIP(c, kf::launch_convert<bf16>(src, reinterpret_cast<bf16*>(c->base + t.off), t.n, c->stream));
      else
        KF_HIP(c, kf::launch_copy_f32(src, reinterpret_cast<float*>(c->base + t.off), t.n, c->stream));
      src += t.n;
    }
    KF_HIP(c, hipMemcpyAsync(c->base + p.omega, omega.data(), omega.size() * 8, hipMemcpyHostToDevice, c->stream));
    if (rmsr)
      KF_HIP(c, hipMemcpyAsync(c->base + p.rope, rope_cs.data(), rope_cs.size() * sizeof(float2),
                               hipMemcpyHostToDevice, c->stream));
    KF_HIP(c, hipStreamSynchronize(c->stream));
  }
  {
    int r = bf ? fold_layernorms<bf16>(c) : fold_layernorms<float>(c);
    if (r) return r;
  }
  // device sequence state starts cleared (context length and error flags)
  KF_HIP(c, kf::launch_zero_i32(reinterpret_cast<int*>(c->base + p.dstate),
                                sizeof(KfDevState) / sizeof(int), c->stream));
  KF_HIP(c, hipStreamSynchronize(c->stream));
  c->weights = true;
  c->live = false;
  c->temp_B = 0;
  return KF_OK;
}

int kf_set_temperature(kf_ctx* c, const float* tau, int B) {
  if (!c) return KF_EINVAL;
  const kf_config& cf = c->cfg;
  if (!(cf.flags & KF_FLAG_TEMPERATURE))
    return fail(c, KF_ESTATE, "the config has no temperature encoder (KF_FLAG_TEMPERATURE)");
  if (B < 1 || B > cf.max_batch) return fail(c, KF_EINVAL, "B=%d outside [1, %d]", B, cf.max_batch);
  if (!tau) return fail(c, KF_EINVAL, "null pointer argument");
  int r = ready(c);
  if (r) return r;
  r = cf.dtype == KF_BF16 ? run_temperature<bf16>(c, tau, B) : run_temperature<float>(c, tau, B);
  if (r) return r;
  c->temp_B = B;
  return KF_OK;
}

int kf_prefill(kf_ctx* c, int B, int N, const int32_t* prompt, int k, const float* noise, int32_t* out) {
  if (!c) return KF_EINVAL;
  const kf_config& cf = c->cfg;
  if (B < 1 || B > cf.max_batch) return fail(c, KF_EINVAL, "B=%d outside [1, %d]", B, cf.max_batch);
  if (N < 0 || N > cf.max_prompt) return fail(c, KF_EINVAL, "N=%d outside [0, %d]", N, cf.max_prompt);
  if (k < 1 || k > cf.max_k) return fail(c, KF_EINVAL, "k=%d outside [1, %d]", k, cf.max_k);
  if (!noise || !out || (N > 0 && !prompt)) return fail(c, KF_EINVAL, "null pointer argument");
  if (N + k > cf.n_ctx) return fail(c, KF_ECTX, "N + k = %d exceeds n_ctx = %d", N + k, cf.n_ctx);
  int r = ready(c);
  if (r) return r;
  r = temp_ready(c, B);
  if (r) return r;
  if ((r = lockstep_begin(c, B))) return r;
  StepIn in{B, N, k, prompt, N, noise, nullptr, 0, out_desc(c, out, k, -1), true};
  r = step(c, in);
  if (r) return r;
  c->live = true;
  c->B = B;
  c->C = N;
  c->pending = k;
  return KF_OK;
}

int kf_decode_block(kf_ctx* c, int B, int k, const float* noise, int32_t* out) {
  if (!c) return KF_EINVAL;
  const kf_config& cf = c->cfg;
  if (k < 1 || k > cf.max_k) return fail(c, KF_EINVAL, "k=%d outside [1, %d]", k, cf.max_k);
  if (!noise || !out) return fail(c, KF_EINVAL, "null pointer argument");
  int r = ready(c);
  if (r) return r;
  r = temp_ready(c, B);
  if (r) return r;
  if (!c->live) return fail(c, KF_ESTATE, "decode before prefill");
  if (B != c->B) return fail(c, KF_ESTATE, "B=%d differs from the prefill's B=%d", B, c->B);
  if (c->C + c->pending + k > cf.n_ctx)
    return fail(c, KF_ECTX, "C + pending + k = %d exceeds n_ctx = %d", c->C + c->pending + k, cf.n_ctx);
  StepIn in{B, c->pending, k, pend_ptr(c), cf.max_k, noise, nullptr, 0, out_desc(c, out, k, -1), false};
  r = step(c, in);
  if (r) return r;
  c->C += c->pending;
  c->pending = k;
  return KF_OK;
}

int kf_decode_block_noalloc(kf_ctx* c, int B, int k, const float* noise, int32_t* out) {
  if (!c) return KF_EINVAL;
  const kf_config& cf = c->cfg;
  if (k < 1 || k > cf.max_k) return fail(c, KF_EINVAL, "k=%d outside [1, %d]", k, cf.max_k);
  if (!noise || !out) return fail(c, KF_EINVAL, "null pointer argument");
  const long long heads = (long long)B * k * c->plan.n_tiles;
  if (heads > KF_NOALLOC_HEAD_ENTRIES)
    return fail(c, KF_EINVAL,
                "B*k*ceil(V/128) = %lld head partials exceed the device scratch maximum of %d "
                "(KF_NOALLOC_HEAD_ENTRIES)",
                heads, KF_NOALLOC_HEAD_ENTRIES);
  int r = ready(c);
  if (r) return r;
  r = temp_ready(c, B);
  if (r) return r;
  if (!c->live) return fail(c, KF_ESTATE, "decode before prefill");
  if (B != c->B) return fail(c, KF_ESTATE, "B=%d differs from the prefill's B=%d", B, c->B);
  if (c->C + c->pending + k > cf.n_ctx)
    return fail(c, KF_ECTX, "C + pending + k = %d exceeds n_ctx = %d", c->C + c->pending + k, cf.n_ctx);
  if (!c->scratch) return fail(c, KF_EHIP, "device scratch unavailable: %s", c->scratch_err.c_str());
  char* b = c->scratch;
  const Scratch scr{reinterpret_cast<float*>(b + kNaAttnM), reinterpret_cast<float*>(b + kNaAttnL),
                    reinterpret_cast<float*>(b + kNaAttnO), KF_NOALLOC_ATTN_ENTRIES,
                    reinterpret_cast<float*>(b + kNaSplit), (size_t)KF_NOALLOC_SPLIT_BYTES,
                    reinterpret_cast<float*>(b + kNaPval), reinterpret_cast<int*>(b + kNaPidx)};
  StepIn in{B, c->pending, k, pend_ptr(c), cf.max_k, noise, nullptr, 0, out_desc(c, out, k, -1), false};
  in.scr = &scr;
  r = step(c, in);
  if (r) return r;
  c->C += c->pending;
  c->pending = k;
  return KF_OK;
}

int kf_generate(kf_ctx* c, int B, int N, const int32_t* prompt, int L, int k, uint64_t seed, int32_t* out) {
  if (!c) return KF_EINVAL;
  const kf_config& cf = c->cfg;
  if (B < 1 || B > cf.max_batch) return fail(c, KF_EINVAL, "B=%d outside [1, %d]", B, cf.max_batch);
  if (N < 0 || N > cf.max_prompt) return fail(c, KF_EINVAL, "N=%d outside [0, %d]", N, cf.max_prompt);
  if (k < 1 || k > cf.max_k) return fail(c, KF_EINVAL, "k=%d outside [1, %d]", k, cf.max_k);
  if (L < 0 || L % k) return fail(c, KF_EINVAL, "L=%d must be a non-negative multiple of k=%d", L, k);
  if (L > 0 && (!out || (N > 0 && !prompt))) return fail(c, KF_EINVAL, "null pointer argument");
  if (N + L > cf.n_ctx) return fail(c, KF_ECTX, "N + L = %d exceeds n_ctx = %d", N + L, cf.n_ctx);
  int r = ready(c);
  if (r) return r;
  r = temp_ready(c, B);
  if (r) return r;
  if (L == 0) return KF_OK;
  if ((r = lockstep_begin(c, B))) return r;
  // The noise rows of every pass (the prefill is pass 0) come from the noise
  // encoder computed ahead, qp passes at a time.
  const Plan& p = c->plan;
  const int passes = L / k, qp = p.nz_rows / (B * k);
  const void* temb = (cf.flags & KF_FLAG_TEMPERATURE) ? c->base + p.temb : nullptr;
  const kf::NoiseAhead na0{reinterpret_cast<const float*>(c->base + p.nz),
                           reinterpret_cast<const float*>(c->base + p.nb2), temb, N, qp, 0};
  if ((r = noise_ahead(c, B, k, N, seed, 0, passes < qp ? passes : qp))) return r;
  StepIn in{B, N, k, prompt, N, nullptr, nullptr, seed, out_desc(c, out, L, N), true};
  in.na = &na0;
  r = step(c, in);
  if (r) return r;
  c->live = true;
  c->B = B;
  c->C = N;
  c->pending = k;
  kf::NoiseAhead nad = na0;
  nad.pass = -1;  // from the committed length
  StepIn dn{B, k, k, pend_ptr(c), cf.max_k, nullptr, nullptr, seed, out_desc(c, out, L, N), false};
  dn.na = &nad;
  return repeat_step(c, dn, passes - 1, k, N, L, [&](int i) {
    if (i % qp) return (int)KF_OK;
    return noise_ahead(c, B, k, N, seed, i, passes - i < qp ? passes - i : qp);
  });
}

int kf_prefill_ar(kf_ctx* c, int B, int N, const int32_t* prompt, const float* u, int32_t* out) {
  if (!c) return KF_EINVAL;
  const kf_config& cf = c->cfg;
  if (B < 1 || B > cf.max_batch) return fail(c, KF_EINVAL, "B=%d outside [1, %d]", B, cf.max_batch);
  if (N < 1 || N > cf.max_prompt) return fail(c, KF_EINVAL, "N=%d outside [1, %d]", N, cf.max_prompt);
  if (!prompt || !u || !out) return fail(c, KF_EINVAL, "null pointer argument");
  if (N + 1 > cf.n_ctx) return fail(c, KF_ECTX, "N + 1 = %d exceeds n_ctx = %d", N + 1, cf.n_ctx);
  int r = ready(c);
  if (r) return r;
  if ((r = lockstep_begin(c, B))) return r;
  StepIn in{B, N, 0, prompt, N, nullptr, u, 0, out_desc(c, out, 1, -1), true};
  r = step(c, in);
  if (r) return r;
  c->live = true;
  c->B = B;
  c->C = N;
  c->pending = 1;
  return KF_OK;
}

int kf_decode_ar(kf_ctx* c, int B, const float* u, int32_t* out) {
  if (!c) return KF_EINVAL;
  const kf_config& cf = c->cfg;
  if (!u || !out) return fail(c, KF_EINVAL, "null pointer argument");
  int r = ready(c);
  if (r) return r;
  if (!c->live) return fail(c, KF_ESTATE, "decode before prefill");
  if (B != c->B) return fail(c, KF_ESTATE, "B=%d differs from the prefill's B=%d", B, c->B);
  if (c->C + c->pending + 1 > cf.n_ctx)
    return fail(c, KF_ECTX, "C + pending + 1 = %d exceeds n_ctx = %d", c->C + c->pending + 1, cf.n_ctx);
  StepIn in{B, c->pending, 0, pend_ptr(c), cf.max_k, nullptr, u, 0, out_desc(c, out, 1, -1), false};
  r = step(c, in);
  if (r) return r;
  c->C += c->pending;
  c->pending = 1;
  return KF_OK;
}

int kf_generate_ar(kf_ctx* c, int B, int N, const int32_t* prompt, int L, uint64_t seed, int32_t* out) {
  if (!c) return KF_EINVAL;
  const kf_config& cf = c->cfg;
  if (B < 1 || B > cf.max_batch) return fail(c, KF_EINVAL, "B=%d outside [1, %d]", B, cf.max_batch);
  if (N < 1 || N > cf.max_prompt) return fail(c, KF_EINVAL, "N=%d outside [1, %d]", N, cf.max_prompt);
  if (L < 0) return fail(c, KF_EINVAL, "L=%d must be >= 0", L);
  if (L > 0 && (!prompt || !out)) return fail(c, KF_EINVAL, "null pointer argument");
  if (N + L > cf.n_ctx) return fail(c, KF_ECTX, "N + L = %d exceeds n_ctx = %d", N + L, cf.n_ctx);
  int r = ready(c);
  if (r) return r;
  if (L == 0) return KF_OK;
  if ((r = lockstep_begin(c, B))) return r;
  StepIn in{B, N, 0, prompt, N, nullptr, nullptr, seed, out_desc(c, out, L, N), true};
  r = step(c, in);
  if (r) return r;
  c->live = true;
  c->B = B;
  c->C = N;
  c->pending = 1;
  StepIn dn{B, 1, 0, pend_ptr(c), cf.max_k, nullptr, nullptr, seed, out_desc(c, out, L, N), false};
  return repeat_step(c, dn, L - 1, 1, N, L);
}

int kf_debug_logits(kf_ctx* c, float* out, size_t n_floats) {
  if (!c) return KF_EINVAL;
  if (!out) return fail(c, KF_EINVAL, "null pointer argument");
  if (!c->base || !c->last_logits) return fail(c, KF_ESTATE, "no logits recorded (needs KF_FLAG_DEBUG_LOGITS and a step)");
  const size_t n = (size_t)c->last_head_rows * c->cfg.vocab;
  if (n_floats < n) return fail(c, KF_EINVAL, "out holds %zu floats, %zu needed", n_floats, n);
  KF_HIP(c, kf::launch_copy_f32(reinterpret_cast<const float*>(c->base + c->plan.logits), out, n, c->stream));
  return KF_OK;
}

int kf_fill_noise(kf_ctx* c, uint64_t seed, int B, int p0, int n, float* out) {
  if (!c) return KF_EINVAL;
  if (B < 1 || n < 1 || p0 < 0 || !out) return fail(c, KF_EINVAL, "bad noise request");
  KF_HIP(c, kf::launch_fill_noise(out, seed, B, p0, n, c->stream));
  return KF_OK;
}

int kf_get_state(const kf_ctx* c, int* C, int* pending, int* B) {
  if (!c) return KF_EINVAL;
  if (C) *C = c->live ? c->C : 0;
  if (pending) *pending = c->live ? c->pending : 0;
  if (B) *B = c->live ? c->B : 0;
  return KF_OK;
}

int kf_device_errors(kf_ctx* c, int* flags) {
  if (!c || !flags) return KF_EINVAL;
  if (!c->base) return fail(c, KF_ESTATE, "no state buffer bound");
  KfDevState h;
  KF_HIP(c, hipStreamSynchronize(c->stream));
  KfDevState* st = reinterpret_cast<KfDevState*>(c->base + c->plan.dstate);
  KF_HIP(c, hipMemcpy(&h, st, sizeof h, hipMemcpyDeviceToHost));
  *flags = h.err;
  if (h.err) KF_HIP(c, kf::launch_zero_i32(&st->err, 1, c->stream));
  KF_HIP(c, hipStreamSynchronize(c->stream));
  return KF_OK;
}

int kf_set_graphs(kf_ctx* c, int enable) {
  if (!c) return KF_EINVAL;
  c->graphs = enable != 0;
  if (!c->graphs) {
    drop_graph(c);
    drop_serve_graphs(c);
  }
  return KF_OK;
}

int kf_set_timing(kf_ctx* c, int class_mask) {
  if (!c) return KF_EINVAL;
  if (class_mask & ~KF_TIMING_ALL) return fail(c, KF_EINVAL, "timing mask 0x%x has unknown bits", class_mask);
  c->timing = class_mask;
  c->ev_used = 0;
  return KF_OK;
}

int kf_kernel_time(kf_ctx* c, int cls, double* total_ms, int* launches) {
  if (!c || !total_ms || !launches) return KF_EINVAL;
  if (cls < 0 || cls >= KF_KC_COUNT) return fail(c, KF_EINVAL, "kernel class %d out of range", cls);
  KF_HIP(c, hipStreamSynchronize(c->stream));
  double tot = 0;
  int n = 0;
  for (size_t i = 0; i < c->ev_used; ++i) {
    if (c->evs[i].cls != cls) continue;
    float ms = 0;
    KF_HIP(c, hipEventElapsedTime(&ms, c->evs[i].a, c->evs[i].b));
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *launches = n;
  return KF_OK;
}

int kf_teacher_targets(kf_ctx* c, int B, int N, const int32_t* tokens, const float* tau,
                       const float* u, int32_t* targets) {
  if (!c) return KF_EINVAL;
  if (int r = ready(c)) return r;
  if (!(c->cfg.flags & KF_FLAG_TEACHER))
    return fail(c, KF_ESTATE, "teacher targets need a context created with KF_FLAG_TEACHER");
  if (B < 1 || B > c->cfg.max_batch) return fail(c, KF_EINVAL, "B = %d outside [1, %d]", B, c->cfg.max_batch);
  if (N < 1 || N > c->cfg.max_prompt)
    return fail(c, KF_EINVAL, "N = %d outside [1, max_prompt = %d]", N, c->cfg.max_prompt);
  if (!tokens || !tau || !u || !targets) return fail(c, KF_EINVAL, "null pointer");
  StepIn in{};
  in.B = B;
  in.nr = N;
  in.k = 0;
  in.toks = tokens;
  in.tok_stride = N;
  in.reset = true;
  in.tau = tau;
  in.u_rows = u;
  in.targets = targets;
  if (int r = lockstep_begin(c, B)) return r;
  // the pass writes the KV cache of every sequence: a generation in progress ends here
  c->live = false;
  c->C = 0;
  c->pending = 0;
  c->B = 0;
  drop_graph(c);
  return step(c, in);
}

int kf_selfforcing_targets(kf_ctx* c, int B, int N, int k, const int32_t* tokens, const float* z1,
                           const float* z2, int32_t* x1, int32_t* x2) {
  if (!c) return KF_EINVAL;
  if (int r = ready(c)) return r;
  const kf_config& cf = c->cfg;
  if (!(cf.flags & KF_FLAG_ROLLOUT))
    return fail(c, KF_ESTATE, "the teacher rollout needs a context created with KF_FLAG_ROLLOUT");
  if (cf.dtype != KF_BF16) return fail(c, KF_EINVAL, "the teacher rollout runs bf16 models only");
  if (B < 1 || B > cf.max_batch) return fail(c, KF_EINVAL, "B = %d outside [1, %d]", B, cf.max_batch);
  if (N < 1 || N > cf.max_prompt)
    return fail(c, KF_EINVAL, "N = %d outside [1, max_prompt = %d]", N, cf.max_prompt);
  if (k < 1 || k > cf.max_k) return fail(c, KF_EINVAL, "k = %d outside [1, max_k = %d]", k, cf.max_k);
  if (N + 2 * k > cf.n_ctx)
    return fail(c, KF_ECTX, "N + 2k = %d exceeds n_ctx = %d", N + 2 * k, cf.n_ctx);
  if (!tokens || !z1 || !z2 || !x1 || !x2) return fail(c, KF_EINVAL, "null pointer");
  if (int r = temp_ready(c, B)) return r;
  // the rollout uses the step workspace and the device state: a generation in progress ends
  c->live = false;
  c->C = 0;
  c->pending = 0;
  c->B = 0;
  drop_graph(c);
  return run_rollout<bf16>(c, B, N, k, tokens, z1, z2, x1, x2);
}

// ------------------------------------------------------ continuous batching
int kf_serve_admit(kf_ctx* c, int n, const int32_t* slots, int N, const int32_t* prompts, int k,
                   const float* noise, int32_t* out) {
  if (!c) return KF_EINVAL;
  const kf_config& cf = c->cfg;
  if (!(cf.flags & KF_FLAG_SERVING)) return fail(c, KF_ESTATE, "serving calls need KF_FLAG_SERVING");
  if (int r = check_slots(c, n, slots)) return r;
  if (N < 0 || N > cf.max_prompt) return fail(c, KF_EINVAL, "N=%d outside [0, %d]", N, cf.max_prompt);
  if (k < 1 || k > cf.max_k) return fail(c, KF_EINVAL, "k=%d outside [1, %d]", k, cf.max_k);
  if (!noise || !out || (N > 0 && !prompts)) return fail(c, KF_EINVAL, "null pointer argument");
  if (N + k > cf.n_ctx) return fail(c, KF_ECTX, "N + k = %d exceeds n_ctx = %d", N + k, cf.n_ctx);
  if (int r = ready(c)) return r;
  int top = 0;
  for (int b = 0; b < n; ++b) {
    if (c->slots.size() != (size_t)cf.max_batch || c->slots[slots[b]].live)
      return fail(c, KF_ESTATE, "slot %d is in use (kf_serve_release it first)", slots[b]);
    top = slots[b] + 1 > top ? slots[b] + 1 : top;
  }
  if (int r = temp_ready(c, top)) return r;
  // admission writes pages the lock-step calls address directly
  c->live = false;
  c->B = c->C = c->pending = 0;
  drop_graph(c);
  std::vector<int> upto(n, N + k);
  if (int r = serve_prepare(c, n, slots, upto)) return r;
  StepIn in{n, N, k, prompts, N, noise, nullptr, 0, out_desc(c, out, k, -1), true};
  in.serve = true;
  for (int b = 0; b < n; ++b) {
    kf_ctx::Slot& sl = c->slots[slots[b]];
    sl.live = true;
    sl.C = N;
    sl.pending = k;
    ++c->serving;
  }
  const int r = step(c, in);
  if (r)
    for (int b = 0; b < n; ++b) serve_free(c, slots[b]);
  return r;
}

int kf_serve_step(kf_ctx* c, int n, const int32_t* slots, int k, const float* noise, int32_t* out) {
  if (!c) return KF_EINVAL;
  const kf_config& cf = c->cfg;
  if (!(cf.flags & KF_FLAG_SERVING)) return fail(c, KF_ESTATE, "serving calls need KF_FLAG_SERVING");
  if (int r = check_slots(c, n, slots)) return r;
  if (k < 1 || k > cf.max_k) return fail(c, KF_EINVAL, "k=%d outside [1, %d]", k, cf.max_k);
  if (!noise || !out) return fail(c, KF_EINVAL, "null pointer argument");
  if (int r = ready(c)) return r;
  if (c->slots.size() != (size_t)cf.max_batch) return fail(c, KF_ESTATE, "no sequence admitted");
  int top = 0, nr = -1;
  std::vector<int> upto(n);
  for (int b = 0; b < n; ++b) {
    const kf_ctx::Slot& sl = c->slots[slots[b]];
    if (!sl.live) return fail(c, KF_ESTATE, "slot %d holds no sequence", slots[b]);
    if (nr >= 0 && sl.pending != nr)
      return fail(c, KF_EINVAL, "slots of one step must have equal pending counts (%d, %d)", nr,
                  sl.pending);
    nr = sl.pending;
    if (sl.C + sl.pending + k > cf.n_ctx)
      return fail(c, KF_ECTX, "slot %d: C + pending + k = %d exceeds n_ctx = %d", slots[b],
                  sl.C + sl.pending + k, cf.n_ctx);
    upto[b] = sl.C + sl.pending + k;
    top = slots[b] + 1 > top ? slots[b] + 1 : top;
  }
  if (int r = temp_ready(c, top)) return r;
  if (int r = serve_prepare(c, n, slots, upto)) return r;
  // On a real stream with timing off, the step replays a graph captured for
  // (n, nr, k): every launch reads the slot map, the committed lengths, the
  // page table and the pending tokens from device memory, and noise and tokens
  // pass through fixed buffers, copied in and out around the replay.
  const bool replay = c->graphs && c->stream != nullptr && !c->timing;
  float* sn = replay ? reinterpret_cast<float*>(c->base + c->plan.serve_noise) : nullptr;
  int32_t* so = replay ? reinterpret_cast<int32_t*>(c->base + c->plan.serve_out) : nullptr;
  StepIn in{n, nr, k, pend_ptr(c), cf.max_k, replay ? sn : noise, nullptr, 0,
            out_desc(c, replay ? so : out, k, -1), false};
  in.serve = true;
  in.toks_by_slot = true;
  if (!replay) {
    if (int r = step(c, in)) return r;
  } else {
    const size_t bytes = (size_t)n * k * 4;
    KF_HIP(c, hipMemcpyAsync(sn, noise, bytes, hipMemcpyDeviceToDevice, c->stream));
    hipGraphExec_t exec = nullptr;
    for (size_t i = 0; i < c->sgraphs.size(); ++i)
      if (c->sgraphs[i].n == n && c->sgraphs[i].nr == nr && c->sgraphs[i].k == k) {
        kf_ctx::ServeGraph g = c->sgraphs[i];
        c->sgraphs.erase(c->sgraphs.begin() + i);
        c->sgraphs.push_back(g);
        exec = g.exec;
        break;
      }
    if (!exec) {
      KF_HIP(c, hipStreamBeginCapture(c->stream, hipStreamCaptureModeRelaxed));
      int r = step(c, in);
      hipGraph_t gr = nullptr;
      hipError_t e = hipStreamEndCapture(c->stream, &gr);
      if (r) {
        if (e == hipSuccess && gr) (void)hipGraphDestroy(gr);
        return r;
      }
      if (e != hipSuccess) return hip_fail(c, e, "hipStreamEndCapture");
      e = hipGraphInstantiate(&exec, gr, nullptr, nullptr, 0);
      (void)hipGraphDestroy(gr);
      if (e != hipSuccess) return hip_fail(c, e, "hipGraphInstantiate");
      if (c->sgraphs.size() == kServeGraphs) {
        (void)hipGraphExecDestroy(c->sgraphs.front().exec);
        c->sgraphs.erase(c->sgraphs.begin());
      }
      c->sgraphs.push_back({n, nr, k, exec});
    }
    KF_HIP(c, hipGraphLaunch(exec, c->stream));
    KF_HIP(c, hipMemcpyAsync(out, so, bytes, hipMemcpyDeviceToDevice, c->stream));
    c->last_head_rows = n * k;  // as the step itself records
    c->last_logits = (cf.flags & KF_FLAG_DEBUG_LOGITS) != 0;
  }
  for (int b = 0; b < n; ++b) {
    kf_ctx::Slot& sl = c->slots[slots[b]];
    sl.C += sl.pending;
    sl.pending = k;
  }
  return KF_OK;
}

int kf_serve_release(kf_ctx* c, int n, const int32_t* slots) {
  if (!c) return KF_EINVAL;
  if (!(c->cfg.flags & KF_FLAG_SERVING)) return fail(c, KF_ESTATE, "serving calls need KF_FLAG_SERVING");
  if (int r = check_slots(c, n, slots)) return r;
  for (int b = 0; b < n; ++b)
    if (c->slots.size() != (size_t)c->cfg.max_batch || !c->slots[slots[b]].live)
      return fail(c, KF_ESTATE, "slot %d holds no sequence", slots[b]);
  for (int b = 0; b < n; ++b) serve_free(c, slots[b]);
  return KF_OK;
}

int kf_serve_state(const kf_ctx* c, int slot, int* C, int* pending, int* pages) {
  if (!c) return KF_EINVAL;
  if (slot < 0 || slot >= c->cfg.max_batch) return KF_EINVAL;
  const bool on = c->slots.size() == (size_t)c->cfg.max_batch && c->slots[slot].live;
  if (C) *C = on ? c->slots[slot].C : -1;
  if (pending) *pending = on ? c->slots[slot].pending : 0;
  if (pages) *pages = on ? (int)c->slots[slot].pages.size() : 0;
  return KF_OK;
}

int kf_serve_pages(const kf_ctx* c, int* free_pages, int* total) {
  if (!c) return KF_EINVAL;
  if (free_pages)
    *free_pages = c->slots.size() == (size_t)c->cfg.max_batch ? (int)c->free_pages.size() : c->plan.n_pages;
  if (total) *total = c->plan.n_pages;
  return KF_OK;
}

int kf_training_attention(void* hip_stream, int mask, int B, int H, int N, int k, int d_head,
                          const void* Q, const void* K, const void* V, void* O, float scale) {
  if (mask != KF_MASK_SINGLE && mask != KF_MASK_DOUBLE) return KF_EINVAL;
  if (B < 0 || H < 0 || N < 0 || k < 1) return KF_EINVAL;
  if (d_head != 32 && d_head != 64 && d_head != 128) return KF_EINVAL;
  if (!isfinite(scale)) return KF_EINVAL;
  if (B == 0 || H == 0 || N == 0) return KF_OK;
  const void* ptrs[4] = {Q, K, V, O};
  for (const void* q : ptrs)
    if (!q || (reinterpret_cast<uintptr_t>(q) & 15)) return KF_EINVAL;
  const int64_t nk = (int64_t)N * k;
  const int64_t rows = mask == KF_MASK_SINGLE ? N + nk : 2 * nk;
  const int64_t keys = mask == KF_MASK_SINGLE ? N + nk : N + 2 * nk;
  const int64_t lim = (int64_t)1 << 31;
  if (keys * d_head >= lim || (int64_t)B * H >= lim || (int64_t)B * H * ((rows + 63) / 64) >= lim)
    return KF_EINVAL;
  const hipError_t e = kf::launch_training_attention(
      mask, B, H, N, k, d_head, static_cast<const bf16*>(Q), static_cast<const bf16*>(K),
      static_cast<const bf16*>(V), static_cast<bf16*>(O), scale,
      static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? KF_OK : KF_EHIP;
}

}  // extern "C"
