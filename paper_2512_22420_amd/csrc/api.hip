// C ABI of the verify step: argument checks, workspace layout, and the kernel
// sequence of one step on one stream (no host synchronisation inside a step).
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/nightjar.h"
#include "attn_work.h"
#include "kernels.h"

using namespace nj;

// Scratch of nightjar_accept_noalloc: a fixed array in device memory, one copy
// per GPU the library runs on, held until the process ends.  In host code this
// name is only a stand-in for the symbol: its device address comes from
// hipGetSymbolAddress (accept_noalloc_scratch below), and only that address is
// ever passed to a kernel.
constexpr size_t kNoAllocScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(NJ_EHIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr size_t kAlign = 256;
constexpr int kMaxK = 15;
constexpr int kMaxVocab = 524288;

size_t al(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }
bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

struct Layout {
  size_t err, gemm_cnt, ctx_snap, attn_cnt, h, x, ssq, rope_cs, qkv, q, win_k, win_v, part_o, part_ml, o, act,
      logits, stats, gemm_part, dacc, dnext, attn_work, total;
  size_t win_layer_bytes;
};

// The step's GEMMs, in order: (N, K, epilogue).
struct GemmShape {
  int N, K, epi;
};
void step_gemms(const nj_model_desc& d, GemmShape out[5]) {
  const int HD = d.n_heads * d.head_dim, QKV = (d.n_heads + 2 * d.n_kv_heads) * d.head_dim;
  out[0] = {QKV, d.d_model, kEpiQkvRope};  // planned as the QKV projection (a streaming plan carries RoPE)
  out[1] = {d.d_model, HD, kEpiResidual};
  out[2] = {2 * d.ffn_dim, d.d_model, kEpiSwiglu};
  out[3] = {d.d_model, d.ffn_dim, kEpiResidual};
  out[4] = {d.vocab, d.d_model, kEpiStore};
}

bool desc_ok(const nj_model_desc* d) {
  if (!d) return !fail(NJ_EINVAL, "desc is NULL");
  if (d->n_layers < 1 || d->d_model < 1 || d->n_heads < 1 || d->n_kv_heads < 1 || d->head_dim < 2 ||
      d->ffn_dim < 1 || d->vocab < 1)
    return !fail(NJ_EINVAL, "model dimensions must be positive");
  if (d->n_heads % d->n_kv_heads) return !fail(NJ_EINVAL, "n_heads %% n_kv_heads != 0");
  if (d->head_dim % 8) return !fail(NJ_EINVAL, "head_dim must be a multiple of 8");
  if (d->block_size != 16) return !fail(NJ_EINVAL, "block_size must be 16");
  if (d->dtype != NJ_F32 && d->dtype != NJ_BF16) return !fail(NJ_EINVAL, "dtype must be NJ_F32 or NJ_BF16");
  if (d->vocab > kMaxVocab) return !fail(NJ_EINVAL, "vocab > %d", kMaxVocab);
  if (!(d->rms_eps >= 0.f) || !(d->rope_theta > 0.f)) return !fail(NJ_EINVAL, "bad rms_eps or rope_theta");
  if (d->d_model % 4 || d->d_model > 8192) return !fail(NJ_EINVAL, "d_model must be a multiple of 4, at most 8192");
  if (d->head_dim > 512) return !fail(NJ_EINVAL, "head_dim > 512");
  if (d->dtype == NJ_BF16) {
    const int qkv = (d->n_heads + 2 * d->n_kv_heads) * d->head_dim;
    if (d->head_dim != 128) return !fail(NJ_EINVAL, "bf16 path needs head_dim 128");
    if (d->d_model % 32 || d->ffn_dim % 32 || (d->n_heads * d->head_dim) % 32)
      return !fail(NJ_EINVAL, "bf16 path needs d_model, ffn_dim, H*D multiples of 32");
    if (qkv % 16 || d->vocab % 16 || d->d_model % 16 || d->ffn_dim % 16)
      return !fail(NJ_EINVAL, "bf16 path needs GEMM output widths (qkv, d, F, V) multiples of 16");
  }
  return true;
}

// Whether a window of M rows runs with the RMSNorms folded into the GEMMs:
// bf16 with every GEMM of the step on the weight-streaming kernel.
// The QKV projection without RoPE in its epilogue (fp32 q/k/v rows for the
// RoPE kernel), on the plan chosen for the QKV projection.
hipError_t launch_qkv_store(int dt, const void* x, const void* w, void* y, int M, int N, int K, int* gcnt, float* gpart,
                            hipStream_t s, bool x_kblocked) {
  if (dt != kBF16) return launch_gemm(dt, x, w, y, M, N, K, kEpiStore, gcnt, gpart, s, x_kblocked);
  return launch_gemm_plan(x, w, y, M, N, K, kEpiStore, gemm_plan(M, N, K, kEpiQkvRope), gcnt, gpart, s, x_kblocked);
}

// Whether a window of M rows runs with the RMSNorms folded into the GEMMs
// (the producer of h writes bf16(h * gain) and per-tile sums of h^2, the
// consumer scales its output rows by 1/rms): bf16, the QKV projection on the
// weight-streaming kernel (RoPE in its epilogue), and each residual GEMM (O,
// down) either streaming or on a tiled plan whose split tiles are reduced by
// all their workgroups (the epilogue that writes the next norm's inputs);
// gate/up and the LM head take the row scale on either kernel.
bool fold_norms(const nj_model_desc& d, int M) {
  if (d.dtype != NJ_BF16 || d.d_model % 32) return false;
  const int HD = d.n_heads * d.head_dim, QKV = (d.n_heads + 2 * d.n_kv_heads) * d.head_dim;
  if (!gemm_streams(M, QKV, d.d_model, kEpiQkvRope)) return false;
  // a tiled consumer reads each row's partials in 16-byte pieces
  const int F2 = 2 * d.ffn_dim;
  if ((!gemm_streams(M, F2, d.d_model, kEpiSwiglu) || !gemm_streams(M, d.vocab, d.d_model, kEpiStore)) &&
      ((d.d_model + 127) / 128) % 4)
    return false;
  auto producer_ok = [&](int K) {
    const GemmPlan p = gemm_plan(M, d.d_model, K, kEpiResidual);
    return p.tile == kTileNone ||
           (p.par && p.part_bytes > 0 && tile_one_segment(p, K) && p.grid <= device_cus());
  };
  return producer_ok(HD) && producer_ok(d.ffn_dim);
}

Layout layout(const nj_model_desc& d, int B, int k) {
  const size_t e = d.dtype == NJ_BF16 ? 2 : 4;
  const size_t T = k + 1, M = (size_t)B * T;
  const size_t HD = (size_t)d.n_heads * d.head_dim;
  const size_t qkv = (size_t)(d.n_heads + 2 * d.n_kv_heads) * d.head_dim;
  const int G = d.n_heads / d.n_kv_heads;
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += al(bytes);
    return o;
  };
  L.err = take(kAlign);
  // Split-K arrival counters of the step's GEMMs: a fixed-size region at a
  // fixed offset, whatever B and k, so that steps of different sizes on one
  // workspace never write activations over them.  Zeroed by
  // nightjar_workspace_init and left at zero by every GEMM.
  L.gemm_cnt = take(kGemmCounterBytes);
  L.ctx_snap = take((size_t)B * 4);  // context lengths read by the verify step, for the KV append
  L.attn_cnt = take((size_t)B * d.n_kv_heads * kCounterStride * 4);  // attention split arrivals (cleared before each launch)
  size_t part = 0;
  if (d.dtype == NJ_BF16) {
    GemmShape gs[5];
    step_gemms(d, gs);
    for (const GemmShape& g : gs) part = std::max(part, gemm_plan((int)M, g.N, g.K, g.epi).part_bytes);
    if (M >= (size_t)kTileMinRows) part = std::max(part, kSplitPartCap);  // any smaller window's plans fit
  }
  L.h = take(M * d.d_model * 4);
  L.x = take(M * d.d_model * e);
  L.ssq = take(M * ((d.d_model + 127) / 128) * 4);  // per-row sums of h^2 over 128-column tiles (folded norm)
  L.rope_cs = take(M * 64 * 2 * 4);                  // the step's RoPE (cos, sin) table (bf16 path)
  L.qkv = take(M * qkv * 4);
  L.q = take(M * HD * e);
  L.win_layer_bytes = (size_t)B * d.n_kv_heads * 16 * d.head_dim * e;
  L.win_k = take(L.win_layer_bytes * d.n_layers);
  L.win_v = take(L.win_layer_bytes * d.n_layers);
  const size_t pf = d.dtype == NJ_BF16 ? attention_partial_floats(B, d.n_kv_heads, (int)T, G, d.head_dim) : 0;
  const size_t pml = pf ? pf / (d.head_dim + 2) * 2 : 0;
  L.part_o = take(pf * 4);
  L.part_ml = take(pml * 4);
  L.o = take(M * HD * e);
  L.act = take(M * d.ffn_dim * e);
  L.logits = take(M * d.vocab * 4);
  L.stats = take(accept_workspace_bytes((int)M, d.vocab));
  L.gemm_part = take(part);  // split-K partials (GEMMs run one after another)
  L.dacc = take((size_t)B * 4);   // draft step: accepted lengths (always 0) and the drawn tokens
  L.dnext = take((size_t)B * 4);
  L.attn_work = take(d.dtype == NJ_BF16 ? attention_work_bytes(B, d.n_kv_heads) : 0);  // built once per step
  L.total = off;
  return L;
}

// Workspace of nightjar_rmsnorm_rope: [error word][split-K counters][x][ssq][rope table][qkv][split-K partials]
struct PreLayout {
  size_t err, gemm_cnt, x, ssq, rope_cs, qkv, gemm_part, total;
};
PreLayout pre_layout(const nj_model_desc& d, int B, int k) {
  const size_t e = d.dtype == NJ_BF16 ? 2 : 4;
  const size_t M = (size_t)B * (k + 1);
  const int QKV = (d.n_heads + 2 * d.n_kv_heads) * d.head_dim;
  PreLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += al(bytes);
    return o;
  };
  L.err = take(kAlign);
  L.gemm_cnt = take(kGemmCounterBytes);
  L.x = take(M * d.d_model * e);
  L.ssq = take(M * ((d.d_model + 127) / 128) * 4);
  L.rope_cs = take(M * 64 * 2 * 4);
  L.qkv = take(M * QKV * 4);
  size_t part = d.dtype == NJ_BF16 ? gemm_plan((int)M, QKV, d.d_model, kEpiQkvRope).part_bytes : 0;
  if (d.dtype == NJ_BF16 && M >= (size_t)kTileMinRows) part = std::max(part, kSplitPartCap);
  L.gemm_part = take(part);
  L.total = off;
  return L;
}

// Workspace of nightjar_attn_verify: [error word][split arrival counters][partial o][partial (m, l)][work list]
struct AttnLayout {
  size_t err, cnt, part_o, part_ml, work, total;
};
AttnLayout attn_layout(const nj_model_desc& d, int B, int k) {
  AttnLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += al(bytes);
    return o;
  };
  L.err = take(kAlign);
  L.cnt = take((size_t)B * d.n_kv_heads * kCounterStride * 4);
  const size_t pf = d.dtype == NJ_BF16
                        ? attention_partial_floats(B, d.n_kv_heads, k + 1, d.n_heads / d.n_kv_heads, d.head_dim)
                        : 0;
  L.part_o = take(pf * 4);
  L.part_ml = take((pf ? pf / (d.head_dim + 2) * 2 : 0) * 4);
  L.work = take(d.dtype == NJ_BF16 ? attention_work_bytes(B, d.n_kv_heads) : 0);
  L.total = off;
  return L;
}

// Device address of `scratch` on each device, taken once per device with
// that device current (the first nightjar_accept_noalloc call on it).
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int accept_noalloc_scratch(void** out);

// Kernel timing of the verify step (nightjar_profile_*): while enabled, each
// launch site of a step records a pair of HIP events on the step's stream;
// reading synchronises the recorded pairs and accumulates their times per
// kernel class.  Event pairs are reused.
struct ProfRec {
  int cls;
  hipEvent_t a, b;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<std::pair<hipEvent_t, hipEvent_t>> g_prof_free;
std::vector<ProfRec> g_prof_pending;
double g_prof_us[NJ_PROF_COUNT] = {};
int64_t g_prof_n[NJ_PROF_COUNT] = {};

struct ProfScope {
  int cls;
  hipStream_t s;
  hipEvent_t a = nullptr, b = nullptr;
  ProfScope(int c, hipStream_t st) : cls(c), s(st) {
    if (!g_prof_on) return;
    std::lock_guard<std::mutex> g(g_prof_mu);
    if (!g_prof_free.empty()) {
      a = g_prof_free.back().first;
      b = g_prof_free.back().second;
      g_prof_free.pop_back();
    } else if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) {
      a = b = nullptr;
      return;
    }
    if (hipEventRecord(a, s) != hipSuccess) a = nullptr;
  }
  ~ProfScope() {
    if (!a || !b) return;
    std::lock_guard<std::mutex> g(g_prof_mu);
    if (hipEventRecord(b, s) == hipSuccess) g_prof_pending.push_back(ProfRec{cls, a, b});
    else g_prof_free.emplace_back(a, b);
  }
};

void prof_drain() {  // caller holds g_prof_mu
  for (const ProfRec& r : g_prof_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      g_prof_us[r.cls] += ms * 1e3;
      ++g_prof_n[r.cls];
    }
    g_prof_free.emplace_back(r.a, r.b);
  }
  g_prof_pending.clear();
}

struct StepRecord {
  int B, k, n_layers;
};
std::mutex g_mu;
std::unordered_map<const void*, StepRecord> g_steps;

int accept_noalloc_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "accept_noalloc: hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(NJ_EINVAL, "accept_noalloc: device id %d out of range", dev);
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "accept_noalloc: hipGetSymbolAddress");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return NJ_OK;
}

}  // namespace

extern "C" {

const char* nightjar_last_error(void) { return g_err.c_str(); }

size_t nightjar_workspace_bytes(const nj_model_desc* desc, int32_t max_B, int32_t max_k) {
  if (!desc_ok(desc) || max_B < 1 || max_k < 0 || max_k > kMaxK) return 0;
  return layout(*desc, max_B, max_k).total;
}

int nightjar_step_folds_norms(const nj_model_desc* desc, int32_t B, int32_t k) {
  if (!desc_ok(desc)) return NJ_EINVAL;
  if (B < 1 || k < 0 || k > kMaxK) return fail(NJ_EINVAL, "bad B or k");
  return fold_norms(*desc, B * (k + 1)) ? 1 : 0;
}

int nightjar_workspace_init(void* workspace, size_t workspace_bytes, void* stream) {
  if (!workspace || workspace_bytes < kAlign) return fail(NJ_EINVAL, "workspace NULL or smaller than %zu", kAlign);
  if (((uintptr_t)workspace & (kAlign - 1)) != 0) return fail(NJ_EINVAL, "workspace must be 256-byte aligned");
  if (workspace_bytes / 4 > (size_t)INT32_MAX) return fail(NJ_EINVAL, "workspace too large");
  hipError_t e = launch_fill_i32(static_cast<int32_t*>(workspace), 0, (int)(workspace_bytes / 4), (hipStream_t)stream);
  return e == hipSuccess ? NJ_OK : hip_fail(e, "workspace_init");
}

int nightjar_device_error(void* workspace, size_t workspace_bytes, void* stream) {
  if (!workspace || workspace_bytes < kAlign) return fail(NJ_EINVAL, "workspace NULL or too small");
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "device_error: stream sync");
  int32_t v = 0;
  e = hipMemcpy(&v, workspace, sizeof v, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "device_error: read");
  if (v) {
    e = launch_fill_i32(static_cast<int32_t*>(workspace), 0, 1, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "device_error: clear");
  }
  return v;
}

}  // extern "C"

namespace {
// Outputs of a draft step (nightjar_draft_step): the drawn token and the
// draft distribution of every sequence, written with strides into the
// target's draft_tokens [B][k] / draft_probs [B][k][V] layout.
struct DraftOut {
  int32_t* tokens;
  int32_t token_stride;
  float* probs;
  int64_t probs_stride;
};

int verify_impl(const nj_model_desc* desc, const nj_weights* w, const nj_kv_cache* kv, const int32_t* block_table,
                int32_t max_blocks, const int32_t* context_lens, const int32_t* last_tokens,
                const int32_t* draft_tokens, const float* draft_probs, const float* uniforms, int32_t B, int32_t k,
                int32_t* accepted_len, int32_t* next_tokens, float* target_logits, void* workspace,
                size_t workspace_bytes, void* stream, const DraftOut* dout) {
  if (!desc_ok(desc)) return NJ_EINVAL;
  const nj_model_desc& d = *desc;
  if (B < 1) return fail(NJ_EINVAL, "B must be >= 1");
  if (k < 0 || k > kMaxK) return fail(NJ_EINVAL, "k must be in [0, %d]", kMaxK);
  if (max_blocks < 1) return fail(NJ_EINVAL, "max_blocks must be >= 1");
  if (!w || !w->embed || !w->final_norm || !w->lm_head || !w->layers) return fail(NJ_EINVAL, "weights incomplete");
  if (!kv || !kv->k_pages || !kv->v_pages || kv->num_blocks < 1) return fail(NJ_EINVAL, "kv cache incomplete");
  if (!block_table || !context_lens || !last_tokens || !uniforms || !accepted_len || !next_tokens || !workspace)
    return fail(NJ_EINVAL, "a required pointer is NULL");
  if (k > 0 && (!draft_tokens || !draft_probs)) return fail(NJ_EINVAL, "k > 0 needs draft_tokens and draft_probs");
  const int T = k + 1, M = B * T, G = d.n_heads / d.n_kv_heads;
  const bool bf = d.dtype == NJ_BF16;
  for (int l = 0; l < d.n_layers; ++l) {
    const nj_layer_weights& lw = w->layers[l];
    if (!lw.attn_norm || !lw.w_qkv || !lw.w_o || !lw.ffn_norm || !lw.w_gate_up || !lw.w_down)
      return fail(NJ_EINVAL, "layer %d weights incomplete", l);
    if (!kv->k_pages[l] || !kv->v_pages[l]) return fail(NJ_EINVAL, "layer %d pages NULL", l);
    if (bf && !(aligned16(lw.w_qkv) && aligned16(lw.w_o) && aligned16(lw.w_gate_up) && aligned16(lw.w_down) &&
                aligned16(kv->k_pages[l]) && aligned16(kv->v_pages[l])))
      return fail(NJ_EINVAL, "layer %d: weights and pages must be 16-byte aligned", l);
  }
  if (bf && !aligned16(w->lm_head)) return fail(NJ_EINVAL, "lm_head must be 16-byte aligned");
  if (target_logits && !aligned16(target_logits)) return fail(NJ_EINVAL, "target_logits must be 16-byte aligned");
  if (bf && T * G > 64) return fail(NJ_EINVAL, "(k+1) * (H/Hkv) = %d exceeds 64 query rows per KV head", T * G);
  if (!bf && (size_t)max_blocks * 16 * 4 > 65536) return fail(NJ_EINVAL, "fp32 path supports max_blocks <= 1024");
  const Layout L = layout(d, B, k);
  if (workspace_bytes < L.total)
    return fail(NJ_EINVAL, "workspace too small: %zu < %zu bytes", workspace_bytes, L.total);
  if (((uintptr_t)workspace & (kAlign - 1)) != 0) return fail(NJ_EINVAL, "workspace must be 256-byte aligned");

  hipStream_t s = (hipStream_t)stream;
  char* ws = static_cast<char*>(workspace);
  int* err = reinterpret_cast<int*>(ws + L.err);
  float* h = reinterpret_cast<float*>(ws + L.h);
  void* x = ws + L.x;
  float* qkv = reinterpret_cast<float*>(ws + L.qkv);
  void* q = ws + L.q;
  void* o = ws + L.o;
  void* act = ws + L.act;
  int* gcnt = reinterpret_cast<int*>(ws + L.gemm_cnt);
  float* gpart = reinterpret_cast<float*>(ws + L.gemm_part);
  float* logits = target_logits ? target_logits : reinterpret_cast<float*>(ws + L.logits);
  const int dt = bf ? kBF16 : kF32;
  const int HD = d.n_heads * d.head_dim, QKV = (d.n_heads + 2 * d.n_kv_heads) * d.head_dim;

  const int attn_wgs = bf ? attention_plan(B, d.n_kv_heads, max_blocks) : 1;

  hipError_t e;
#define NJ_TRY(cls, call, what)                    \
  do {                                             \
    ProfScope prof_(cls, s);                       \
    e = (call);                                    \
    if (e != hipSuccess) return hip_fail(e, what); \
  } while (0)

  // bf16 with every GEMM on the weight-streaming kernel: the RMSNorms are
  // folded into the GEMMs (the residual GEMMs and the embedding write h * gain
  // and per-tile sums of h^2; the next GEMM scales its rows by 1/rms)
  const int F2 = 2 * d.ffn_dim;
  bool fused = fold_norms(d, M) && aligned16(w->final_norm);
  for (int l = 0; l < d.n_layers && fused; ++l)
    fused = aligned16(w->layers[l].attn_norm) && aligned16(w->layers[l].ffn_norm);
  // Without the folded norm, the input of each GEMM that runs on the
  // LDS-tiled kernel is written k-blocked by its producer (norm, attention,
  // SwiGLU epilogue), so the tile loads read 1 KB contiguous units.
  const bool kb_qkv = bf && !gemm_streams(M, QKV, d.d_model, kEpiQkvRope);
  const bool kb_o = bf && !gemm_streams(M, d.d_model, HD, kEpiResidual);
  const bool kb_gu = bf && !gemm_streams(M, F2, d.d_model, kEpiSwiglu);
  const bool kb_dn = bf && d.ffn_dim % 32 == 0 && !gemm_streams(M, d.d_model, d.ffn_dim, kEpiResidual);
  const bool kb_lm = bf && !gemm_streams(M, d.vocab, d.d_model, kEpiStore);
  float* ssq = reinterpret_cast<float*>(ws + L.ssq);
  const int nt = (d.d_model + 127) / 128;
  const GemmNorm scale_in{ssq, nt, d.rms_eps, nullptr, nullptr, nullptr, nullptr};

  // the embedding kernel carries one more workgroup that builds the
  // attention's work list for every layer of the step (bf16)
  const AttnPlan plan{context_lens, reinterpret_cast<AttnWork*>(ws + L.attn_work), B, d.n_kv_heads, T, max_blocks,
                      attn_wgs, bf && attention_orders(attn_wgs) ? 1 : 0};
  const AttnPlan* pl = bf ? &plan : nullptr;
  // Norms not folded, but a QKV GEMM that still streams: RoPE and the window
  // store in its epilogue (no row scale), from the table the embedding kernel writes
  const bool rope_in_qkv = !fused && bf && gemm_streams(M, QKV, d.d_model, kEpiQkvRope);
  if (fused)
    NJ_TRY(NJ_PROF_EMBED, launch_embed_gather(last_tokens, draft_tokens, B, T, w->embed, w->layers[0].attn_norm, h, x, ssq, d.d_model,
                               d.vocab, err, context_lens, d.rope_theta, reinterpret_cast<float*>(ws + L.rope_cs), s, pl),
           "embed");
  else
    NJ_TRY(NJ_PROF_EMBED, launch_embed_norm(dt, last_tokens, draft_tokens, B, T, w->embed, w->layers[0].attn_norm, h, x, d.d_model,
                             d.vocab, d.rms_eps, err, s, kb_qkv, pl, context_lens, d.rope_theta,
                             rope_in_qkv ? reinterpret_cast<float*>(ws + L.rope_cs) : nullptr),
           "embed");
  for (int l = 0; l < d.n_layers; ++l) {
    const nj_layer_weights& lw = w->layers[l];
    void* wk = ws + L.win_k + l * L.win_layer_bytes;
    void* wv = ws + L.win_v + l * L.win_layer_bytes;
    int32_t* snap = l == 0 ? reinterpret_cast<int32_t*>(ws + L.ctx_snap) : nullptr;
    int* acnt = bf ? reinterpret_cast<int*>(ws + L.attn_cnt) : nullptr;
    if (fused) {  // RoPE and the window store in the QKV GEMM's epilogue
      const QkvRope rope{context_lens, T, d.n_heads, d.n_kv_heads, reinterpret_cast<const float*>(ws + L.rope_cs), q,
                         wk, wv, snap, acnt};
      NJ_TRY(NJ_PROF_QKV, launch_gemm_norm(x, lw.w_qkv, qkv, M, QKV, d.d_model, kEpiQkvRope, scale_in, gcnt, gpart, s, &rope),
             "qkv gemm");
    } else {
      if (l > 0) NJ_TRY(NJ_PROF_NORM, launch_rmsnorm(dt, h, lw.attn_norm, x, M, d.d_model, d.rms_eps, s, kb_qkv), "attn_norm");
      if (rope_in_qkv) {
        const QkvRope rope{context_lens, T, d.n_heads, d.n_kv_heads, reinterpret_cast<const float*>(ws + L.rope_cs), q,
                           wk, wv, snap, acnt};
        const GemmNorm unscaled{nullptr, 0, 0.f, nullptr, nullptr, nullptr, nullptr};
        NJ_TRY(NJ_PROF_QKV, launch_gemm_norm(x, lw.w_qkv, qkv, M, QKV, d.d_model, kEpiQkvRope, unscaled, gcnt, gpart, s, &rope),
               "qkv gemm");
      } else {
        NJ_TRY(NJ_PROF_QKV, launch_qkv_store(dt, x, lw.w_qkv, qkv, M, QKV, d.d_model, gcnt, gpart, s, kb_qkv), "qkv gemm");
        NJ_TRY(NJ_PROF_ROPE, launch_rope_window(dt, qkv, context_lens, B, T, d.n_heads, d.n_kv_heads, d.head_dim, d.rope_theta, q,
                                  wk, wv, snap, acnt, s),
               "rope");
      }
    }
    AttnArgs aa{dt, q, kv->k_pages[l], kv->v_pages[l], wk, wv, block_table, max_blocks, context_lens,
                kv->num_blocks, B, T, d.n_heads, d.n_kv_heads, d.head_dim,
                reinterpret_cast<float*>(ws + L.part_o), reinterpret_cast<float*>(ws + L.part_ml),
                reinterpret_cast<int*>(ws + L.attn_cnt), attn_wgs, reinterpret_cast<const AttnWork*>(ws + L.attn_work), o,
                err, kb_o};
    NJ_TRY(NJ_PROF_ATTENTION, launch_attention(aa, s), "attention");
    const void* g_next = l + 1 < d.n_layers ? w->layers[l + 1].attn_norm : w->final_norm;
    if (fused) {
      // each input in the layout its consumer's kernel reads (k-blocked for a tiled plan)
      const GemmNorm to_ffn{nullptr, 0, 0.f, lw.ffn_norm, x, ssq, nullptr, kb_gu};
      NJ_TRY(NJ_PROF_O, launch_gemm_norm(o, lw.w_o, h, M, d.d_model, HD, kEpiResidualNorm, to_ffn, gcnt, gpart, s, nullptr, kb_o),
             "o gemm");
      NJ_TRY(NJ_PROF_GATE_UP, launch_gemm_norm(x, lw.w_gate_up, act, M, F2, d.d_model, kEpiSwiglu, scale_in, gcnt, gpart, s,
                                               nullptr, kb_gu, kb_dn),
             "gate_up gemm");
      const GemmNorm to_next{nullptr, 0, 0.f, g_next, x, ssq, nullptr, l + 1 < d.n_layers ? kb_qkv : kb_lm};
      NJ_TRY(NJ_PROF_DOWN, launch_gemm_norm(act, lw.w_down, h, M, d.d_model, d.ffn_dim, kEpiResidualNorm, to_next, gcnt, gpart,
                                            s, nullptr, kb_dn),
             "down gemm");
    } else {
      NJ_TRY(NJ_PROF_O, launch_gemm(dt, o, lw.w_o, h, M, d.d_model, HD, kEpiResidual, gcnt, gpart, s, kb_o), "o gemm");
      NJ_TRY(NJ_PROF_NORM, launch_rmsnorm(dt, h, lw.ffn_norm, x, M, d.d_model, d.rms_eps, s, kb_gu), "ffn_norm");
      NJ_TRY(NJ_PROF_GATE_UP, launch_gemm(dt, x, lw.w_gate_up, act, M, F2, d.d_model, kEpiSwiglu, gcnt, gpart, s, kb_gu, kb_dn),
             "gate_up gemm");
      NJ_TRY(NJ_PROF_DOWN, launch_gemm(dt, act, lw.w_down, h, M, d.d_model, d.ffn_dim, kEpiResidual, gcnt, gpart, s, kb_dn),
             "down gemm");
    }
  }
  bool stats_ready = false;
  float* stats = accept_stats_ptr(ws + L.stats);
  if (fused) {
    const GemmNorm lm{ssq, nt, d.rms_eps, nullptr, nullptr, nullptr, stats};
    NJ_TRY(NJ_PROF_LM_HEAD, launch_gemm_norm(x, w->lm_head, logits, M, d.vocab, d.d_model, kEpiLogits, lm, gcnt, gpart, s,
                                             nullptr, kb_lm),
           "lm_head gemm");
    stats_ready = true;
  } else {
    NJ_TRY(NJ_PROF_NORM, launch_rmsnorm(dt, h, w->final_norm, x, M, d.d_model, d.rms_eps, s, kb_lm), "final_norm");
    if (bf)
      NJ_TRY(NJ_PROF_LM_HEAD, launch_gemm_logits(x, w->lm_head, logits, stats, M, d.vocab, d.d_model, gcnt, gpart, s, &stats_ready,
                                kb_lm),
             "lm_head gemm");
    else
      NJ_TRY(NJ_PROF_LM_HEAD, launch_gemm(dt, x, w->lm_head, logits, M, d.vocab, d.d_model, kEpiStore, gcnt, gpart, s), "lm_head gemm");
  }
  AcceptArgs ac{logits, draft_tokens, draft_probs, uniforms, B, k, d.vocab, ws + L.stats, stats_ready,
                stats_ready ? logits_stat_entries(M, d.vocab, d.d_model) : 0, accepted_len, next_tokens, err};
  NJ_TRY(NJ_PROF_ACCEPT, launch_accept(ac, s), "accept");
  if (dout)
    NJ_TRY(NJ_PROF_ACCEPT, launch_emit_draft(ac, dout->tokens, dout->token_stride, dout->probs, dout->probs_stride, s),
           "emit draft");
#undef NJ_TRY
  {
    std::lock_guard<std::mutex> g(g_mu);
    g_steps[workspace] = StepRecord{B, k, d.n_layers};
  }
  return NJ_OK;
}

}  // namespace

extern "C" {

int nightjar_verify_step(const nj_model_desc* desc, const nj_weights* w, const nj_kv_cache* kv,
                         const int32_t* block_table, int32_t max_blocks, const int32_t* context_lens,
                         const int32_t* last_tokens, const int32_t* draft_tokens, const float* draft_probs,
                         const float* uniforms, int32_t B, int32_t k, int32_t* accepted_len, int32_t* next_tokens,
                         float* target_logits, void* workspace, size_t workspace_bytes, void* stream) {
  return verify_impl(desc, w, kv, block_table, max_blocks, context_lens, last_tokens, draft_tokens, draft_probs,
                     uniforms, B, k, accepted_len, next_tokens, target_logits, workspace, workspace_bytes, stream,
                     nullptr);
}

int nightjar_draft_step(const nj_model_desc* desc, const nj_weights* w, const nj_kv_cache* kv,
                        const int32_t* block_table, int32_t max_blocks, const int32_t* context_lens,
                        const int32_t* last_tokens, const float* uniforms, int32_t B, int32_t* token_out,
                        int32_t token_stride, float* probs_out, int64_t probs_stride, void* workspace,
                        size_t workspace_bytes, void* stream) {
  if (!desc_ok(desc)) return NJ_EINVAL;
  if (B < 1) return fail(NJ_EINVAL, "B must be >= 1");
  if (!token_out || !probs_out || !workspace) return fail(NJ_EINVAL, "a required pointer is NULL");
  if (token_stride < 1 || probs_stride < desc->vocab)
    return fail(NJ_EINVAL, "token_stride must be >= 1 and probs_stride >= vocab");
  if (((uintptr_t)workspace & (kAlign - 1)) != 0) return fail(NJ_EINVAL, "workspace must be 256-byte aligned");
  const Layout L = layout(*desc, B, 0);
  if (workspace_bytes < L.total) return fail(NJ_EINVAL, "workspace too small: %zu < %zu bytes", workspace_bytes, L.total);
  char* ws = static_cast<char*>(workspace);
  const DraftOut dout{token_out, token_stride, probs_out, probs_stride};
  return verify_impl(desc, w, kv, block_table, max_blocks, context_lens, last_tokens, nullptr, nullptr, uniforms, B, 0,
                     reinterpret_cast<int32_t*>(ws + L.dacc), reinterpret_cast<int32_t*>(ws + L.dnext), nullptr,
                     workspace, workspace_bytes, stream, &dout);
}

size_t nightjar_sd_workspace_bytes(const nj_model_desc* draft, int32_t B) {
  if (!desc_ok(draft) || B < 1) return 0;
  // the draft's own step workspace, then its context lengths during the
  // chain, a scratch token and a scratch distribution for the catch-up forward
  return layout(*draft, B, 0).total + al((size_t)B * 4) * 4 + al((size_t)B * draft->vocab * 4);
}

int nightjar_sd_step(const nj_model_desc* target, const nj_weights* tw, const nj_kv_cache* tkv,
                     const nj_model_desc* draft, const nj_weights* dw, const nj_kv_cache* dkv,
                     const int32_t* block_table, int32_t max_blocks, int32_t* context_lens,
                     const int32_t* last_tokens, const float* draft_uniforms, const float* uniforms, int32_t B,
                     int32_t k, int32_t* draft_tokens, float* draft_probs, int32_t* accepted_len,
                     int32_t* next_tokens, void* target_ws, size_t target_ws_bytes, void* draft_ws,
                     size_t draft_ws_bytes, void* stream) {
  if (!desc_ok(target) || !desc_ok(draft)) return NJ_EINVAL;
  if (target->vocab != draft->vocab) return fail(NJ_EINVAL, "draft and target vocabularies differ");
  if (B < 1 || k < 0 || k > kMaxK) return fail(NJ_EINVAL, "bad B or k");
  if (k > 0 && (!draft_tokens || !draft_probs || !draft_uniforms || !dw || !dkv || !draft_ws))
    return fail(NJ_EINVAL, "k > 0 needs the draft model, its cache, workspace, uniforms and outputs");
  const int V = target->vocab;
  hipStream_t s = (hipStream_t)stream;
  int rc;
  if (k > 0) {
    const size_t need = nightjar_sd_workspace_bytes(draft, B);
    if (draft_ws_bytes < need) return fail(NJ_EINVAL, "draft workspace too small: %zu < %zu", draft_ws_bytes, need);
    if (((uintptr_t)draft_ws & (kAlign - 1)) != 0) return fail(NJ_EINVAL, "workspace must be 256-byte aligned");
    char* ws = static_cast<char*>(draft_ws);
    const size_t base = layout(*draft, B, 0).total;
    const size_t b4 = al((size_t)B * 4);
    int32_t* dctx = reinterpret_cast<int32_t*>(ws + base);
    int32_t* tok_in = reinterpret_cast<int32_t*>(ws + base + b4);
    int32_t* tok_scratch = reinterpret_cast<int32_t*>(ws + base + 2 * b4);
    float* u_in = reinterpret_cast<float*>(ws + base + 3 * b4);
    float* prob_scratch = reinterpret_cast<float*>(ws + base + 4 * b4);
    const int32_t* dacc = reinterpret_cast<const int32_t*>(ws + layout(*draft, B, 0).dacc);
    hipError_t e = launch_copy_i32(dctx, context_lens, B, s);  // the draft cache is in step with the target's
    if (e != hipSuccess) return hip_fail(e, "sd_step: draft context");
    // the draft chain: forward i takes the previous token, draws draft i+1 and
    // records q_i; forward k only commits draft k's KV (its draw is not used),
    // so the draft cache never falls behind the target's
    for (int i = 0; i <= k; ++i) {
      // this forward's input token and uniform, gathered from their columns
      e = launch_gather_u32(tok_in, i == 0 ? last_tokens : draft_tokens + (i - 1), B, i == 0 ? 1 : k, s);
      if (e == hipSuccess)
        e = launch_gather_u32(reinterpret_cast<int32_t*>(u_in), reinterpret_cast<const int32_t*>(draft_uniforms) + i,
                              B, k + 1, s);
      if (e != hipSuccess) return hip_fail(e, "sd_step: gather");
      rc = nightjar_draft_step(draft, dw, dkv, block_table, max_blocks, dctx, tok_in, u_in, B,
                               i < k ? draft_tokens + i : tok_scratch, i < k ? k : 1,
                               i < k ? draft_probs + (size_t)i * V : prob_scratch, i < k ? (int64_t)k * V : (int64_t)V,
                               draft_ws, draft_ws_bytes, stream);
      if (rc != NJ_OK) return rc;
      rc = nightjar_kv_append(draft, dkv, block_table, max_blocks, dctx, dacc, B, 0, draft_ws, draft_ws_bytes, stream);
      if (rc != NJ_OK) return rc;
    }
  }
  rc = nightjar_verify_step(target, tw, tkv, block_table, max_blocks, context_lens, last_tokens, draft_tokens,
                            draft_probs, uniforms, B, k, accepted_len, next_tokens, nullptr, target_ws, target_ws_bytes,
                            stream);
  if (rc != NJ_OK) return rc;
  return nightjar_kv_append(target, tkv, block_table, max_blocks, context_lens, accepted_len, B, k, target_ws,
                            target_ws_bytes, stream);
}

int nightjar_kv_append(const nj_model_desc* desc, const nj_kv_cache* kv, const int32_t* block_table,
                       int32_t max_blocks, int32_t* context_lens, const int32_t* accepted_len, int32_t B, int32_t k,
                       const void* workspace, size_t workspace_bytes, void* stream) {
  if (!desc_ok(desc)) return NJ_EINVAL;
  const nj_model_desc& d = *desc;
  if (!kv || !kv->k_pages || !kv->v_pages || kv->num_blocks < 1) return fail(NJ_EINVAL, "kv cache incomplete");
  if (!block_table || !context_lens || !accepted_len || !workspace) return fail(NJ_EINVAL, "a required pointer is NULL");
  if (B < 1 || k < 0 || k > kMaxK || max_blocks < 1) return fail(NJ_EINVAL, "bad B, k or max_blocks");
  for (int l = 0; l < d.n_layers; ++l)
    if (!kv->k_pages[l] || !kv->v_pages[l]) return fail(NJ_EINVAL, "layer %d pages NULL", l);
  {
    std::lock_guard<std::mutex> g(g_mu);
    auto it = g_steps.find(workspace);
    if (it == g_steps.end()) return fail(NJ_EINVAL, "no verify step has filled this workspace");
    if (it->second.B != B || it->second.k != k || it->second.n_layers != d.n_layers)
      return fail(NJ_EINVAL, "B/k/layers differ from the verify step that filled the workspace");
  }
  const Layout L = layout(d, B, k);
  if (workspace_bytes < L.total) return fail(NJ_EINVAL, "workspace too small");
  const char* ws = static_cast<const char*>(workspace);
  for (int l = 0; l < d.n_layers; ++l)
    if (!aligned16(kv->k_pages[l]) || !aligned16(kv->v_pages[l])) return fail(NJ_EINVAL, "layer %d pages not 16-byte aligned", l);
  KvAppendArgs a{d.dtype == NJ_BF16 ? kBF16 : kF32, kv->k_pages, kv->v_pages, ws + L.win_k, ws + L.win_v,
                 block_table, max_blocks, kv->num_blocks, reinterpret_cast<const int32_t*>(ws + L.ctx_snap),
                 context_lens, accepted_len, d.n_layers, B, k, d.n_kv_heads, d.head_dim,
                 reinterpret_cast<int*>(const_cast<char*>(ws) + L.err)};
  hipError_t e;
  {
    ProfScope prof_(NJ_PROF_KV_APPEND, (hipStream_t)stream);
    e = launch_kv_append(a, (hipStream_t)stream);
  }
  return e == hipSuccess ? NJ_OK : hip_fail(e, "kv_append");
}

int nightjar_profile_enable(int32_t enable) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  prof_drain();
  for (int c = 0; c < NJ_PROF_COUNT; ++c) {
    g_prof_us[c] = 0.0;
    g_prof_n[c] = 0;
  }
  g_prof_on = enable != 0;
  return NJ_OK;
}

int nightjar_profile_read(int32_t kernel, double* mean_us, int64_t* launches) {
  if (kernel < 0 || kernel >= NJ_PROF_COUNT || !mean_us || !launches)
    return fail(NJ_EINVAL, "profile_read: bad kernel class or NULL output");
  std::lock_guard<std::mutex> g(g_prof_mu);
  prof_drain();
  *launches = g_prof_n[kernel];
  *mean_us = g_prof_n[kernel] ? g_prof_us[kernel] / (double)g_prof_n[kernel] : 0.0;
  return NJ_OK;
}

size_t nightjar_rmsnorm_rope_workspace_bytes(const nj_model_desc* desc, int32_t B, int32_t k) {
  if (!desc_ok(desc)) return 0;
  if (B < 1 || k < 0 || k > kMaxK) {
    fail(NJ_EINVAL, "bad B or k");
    return 0;
  }
  return pre_layout(*desc, B, k).total;
}

int nightjar_rmsnorm_rope(const nj_model_desc* desc, const float* h, const void* attn_norm, const void* w_qkv,
                          const int32_t* context_lens, int32_t B, int32_t k, void* q_out, void* win_k, void* win_v,
                          void* workspace, size_t workspace_bytes, void* stream) {
  if (!desc_ok(desc)) return NJ_EINVAL;
  const nj_model_desc& d = *desc;
  if (B < 1 || k < 0 || k > kMaxK) return fail(NJ_EINVAL, "bad B or k");
  if (!h || !attn_norm || !w_qkv || !context_lens || !q_out || !win_k || !win_v || !workspace)
    return fail(NJ_EINVAL, "a required pointer is NULL");
  const bool bf = d.dtype == NJ_BF16;
  if (!(aligned16(h) && aligned16(attn_norm) && aligned16(w_qkv) && aligned16(q_out) && aligned16(win_k) &&
        aligned16(win_v)))
    return fail(NJ_EINVAL, "h, attn_norm, w_qkv, q_out, win_k and win_v must be 16-byte aligned");
  const PreLayout L = pre_layout(d, B, k);
  if (workspace_bytes < L.total) return fail(NJ_EINVAL, "workspace too small: %zu < %zu bytes", workspace_bytes, L.total);
  if (((uintptr_t)workspace & (kAlign - 1)) != 0) return fail(NJ_EINVAL, "workspace must be 256-byte aligned");
  const int T = k + 1, M = B * T, QKV = (d.n_heads + 2 * d.n_kv_heads) * d.head_dim;
  const int dt = bf ? kBF16 : kF32;
  hipStream_t s = (hipStream_t)stream;
  char* ws = static_cast<char*>(workspace);
  int* gcnt = reinterpret_cast<int*>(ws + L.gemm_cnt);
  float* gpart = reinterpret_cast<float*>(ws + L.gemm_part);
  float* ssq = reinterpret_cast<float*>(ws + L.ssq);
  float* cs = reinterpret_cast<float*>(ws + L.rope_cs);
  hipError_t e;
  if (fold_norms(d, M)) {  // the step's kernels for this window: norm folded into the QKV GEMM, RoPE in its epilogue
    e = launch_norm_inputs(h, B, T, attn_norm, ws + L.x, ssq, d.d_model, context_lens, d.rope_theta, cs, s);
    if (e != hipSuccess) return hip_fail(e, "rmsnorm_rope: norm inputs");
    const GemmNorm scale_in{ssq, (d.d_model + 127) / 128, d.rms_eps, nullptr, nullptr, nullptr, nullptr};
    const QkvRope rope{context_lens, T, d.n_heads, d.n_kv_heads, cs, q_out, win_k, win_v, nullptr, nullptr};
    e = launch_gemm_norm(ws + L.x, w_qkv, ws + L.qkv, M, QKV, d.d_model, kEpiQkvRope, scale_in, gcnt, gpart, s, &rope);
    return e == hipSuccess ? NJ_OK : hip_fail(e, "rmsnorm_rope: qkv gemm");
  }
  const bool kb = bf && !gemm_streams(M, QKV, d.d_model, kEpiQkvRope);
  e = launch_rmsnorm(dt, h, attn_norm, ws + L.x, M, d.d_model, d.rms_eps, s, kb);
  if (e == hipSuccess) e = launch_qkv_store(dt, ws + L.x, w_qkv, ws + L.qkv, M, QKV, d.d_model, gcnt, gpart, s, kb);
  if (e == hipSuccess)
    e = launch_rope_window(dt, reinterpret_cast<const float*>(ws + L.qkv), context_lens, B, T, d.n_heads,
                           d.n_kv_heads, d.head_dim, d.rope_theta, q_out, win_k, win_v, nullptr, nullptr, s);
  return e == hipSuccess ? NJ_OK : hip_fail(e, "rmsnorm_rope");
}

size_t nightjar_attn_workspace_bytes(const nj_model_desc* desc, int32_t B, int32_t k) {
  if (!desc_ok(desc)) return 0;
  if (B < 1 || k < 0 || k > kMaxK) {
    fail(NJ_EINVAL, "bad B or k");
    return 0;
  }
  return attn_layout(*desc, B, k).total;
}

int nightjar_attn_verify(const nj_model_desc* desc, const void* q, const void* k_pages, const void* v_pages,
                         int32_t num_blocks, const void* win_k, const void* win_v, const int32_t* block_table,
                         int32_t max_blocks, const int32_t* context_lens, int32_t B, int32_t k, void* out,
                         void* workspace, size_t workspace_bytes, void* stream) {
  if (!desc_ok(desc)) return NJ_EINVAL;
  const nj_model_desc& d = *desc;
  if (B < 1 || k < 0 || k > kMaxK) return fail(NJ_EINVAL, "bad B or k");
  if (max_blocks < 1 || num_blocks < 1) return fail(NJ_EINVAL, "max_blocks and num_blocks must be >= 1");
  if (!q || !k_pages || !v_pages || !win_k || !win_v || !block_table || !context_lens || !out || !workspace)
    return fail(NJ_EINVAL, "a required pointer is NULL");
  const bool bf = d.dtype == NJ_BF16;
  const int T = k + 1, G = d.n_heads / d.n_kv_heads;
  if (bf && !(aligned16(q) && aligned16(k_pages) && aligned16(v_pages) && aligned16(win_k) && aligned16(win_v) &&
              aligned16(out)))
    return fail(NJ_EINVAL, "q, pages, window blocks and out must be 16-byte aligned");
  if (bf && T * G > 64) return fail(NJ_EINVAL, "(k+1) * (H/Hkv) = %d exceeds 64 query rows per KV head", T * G);
  if (!bf && (size_t)max_blocks * 16 * 4 > 65536) return fail(NJ_EINVAL, "fp32 path supports max_blocks <= 1024");
  const AttnLayout L = attn_layout(d, B, k);
  if (workspace_bytes < L.total) return fail(NJ_EINVAL, "workspace too small: %zu < %zu bytes", workspace_bytes, L.total);
  if (((uintptr_t)workspace & (kAlign - 1)) != 0) return fail(NJ_EINVAL, "workspace must be 256-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  char* ws = static_cast<char*>(workspace);
  int* cnt = reinterpret_cast<int*>(ws + L.cnt);
  hipError_t e = hipSuccess;
  const int wgs = bf ? attention_plan(B, d.n_kv_heads, max_blocks) : 1;
  // the work list, with the split arrival counters cleared
  if (bf) e = launch_attn_plan(context_lens, B, d.n_kv_heads, T, max_blocks, wgs, ws + L.work, cnt, s);
  if (e != hipSuccess) return hip_fail(e, "attn_verify: work list");
  AttnArgs aa{bf ? kBF16 : kF32, q, k_pages, v_pages, win_k, win_v, block_table, max_blocks, context_lens,
              num_blocks, B, T, d.n_heads, d.n_kv_heads, d.head_dim,
              reinterpret_cast<float*>(ws + L.part_o), reinterpret_cast<float*>(ws + L.part_ml), cnt, wgs,
              reinterpret_cast<const AttnWork*>(ws + L.work), out, reinterpret_cast<int*>(ws + L.err), false};
  e = launch_attention(aa, s);
  return e == hipSuccess ? NJ_OK : hip_fail(e, "attn_verify");
}

size_t nightjar_accept_workspace_bytes(int32_t vocab, int32_t B, int32_t k) {
  if (vocab < 1 || vocab > kMaxVocab || B < 1 || k < 0 || k > kMaxK) {
    fail(NJ_EINVAL, "bad vocab, B or k");
    return 0;
  }
  return kAlign + accept_workspace_bytes(B * (k + 1), vocab);
}

int nightjar_accept(const nj_model_desc* desc, const float* logits, const int32_t* draft_tokens,
                    const float* draft_probs, const float* uniforms, int32_t B, int32_t k, int32_t* accepted_len,
                    int32_t* next_tokens, void* workspace, size_t workspace_bytes, void* stream) {
  if (!desc || desc->vocab < 1 || desc->vocab > kMaxVocab) return fail(NJ_EINVAL, "bad desc or vocab");
  if (B < 1 || k < 0 || k > kMaxK) return fail(NJ_EINVAL, "bad B or k");
  if (!logits || !uniforms || !accepted_len || !next_tokens || !workspace)
    return fail(NJ_EINVAL, "a required pointer is NULL");
  if (k > 0 && (!draft_tokens || !draft_probs)) return fail(NJ_EINVAL, "k > 0 needs draft_tokens and draft_probs");
  const size_t need = nightjar_accept_workspace_bytes(desc->vocab, B, k);
  if (workspace_bytes < need) return fail(NJ_EINVAL, "workspace too small: %zu < %zu", workspace_bytes, need);
  if (((uintptr_t)workspace & (kAlign - 1)) != 0) return fail(NJ_EINVAL, "workspace must be 256-byte aligned");
  char* ws = static_cast<char*>(workspace);
  AcceptArgs a{logits, draft_tokens, draft_probs, uniforms, B, k, desc->vocab, ws + kAlign, false, 0, accepted_len,
               next_tokens, reinterpret_cast<int*>(ws)};
  hipError_t e = launch_accept(a, (hipStream_t)stream);
  return e == hipSuccess ? NJ_OK : hip_fail(e, "accept");
}

int nightjar_accept_noalloc(const nj_model_desc* desc, const float* logits, const int32_t* draft_tokens,
                            const float* draft_probs, const float* uniforms, int32_t B, int32_t k,
                            int32_t* accepted_len, int32_t* next_tokens, int32_t* device_error, void* stream) {
  if (!desc || desc->vocab < 1 || desc->vocab > kMaxVocab) return fail(NJ_EINVAL, "bad desc or vocab");
  if (B < 1 || k < 0 || k > kMaxK) return fail(NJ_EINVAL, "bad B or k");
  if (!logits || !uniforms || !accepted_len || !next_tokens || !device_error)
    return fail(NJ_EINVAL, "a required pointer is NULL");
  if (k > 0 && (!draft_tokens || !draft_probs)) return fail(NJ_EINVAL, "k > 0 needs draft_tokens and draft_probs");
  const size_t need = accept_workspace_bytes(B * (k + 1), desc->vocab);
  if (need > kNoAllocScratchBytes)
    return fail(NJ_EINVAL, "accept_noalloc: B=%d, k=%d, vocab=%d needs %zu bytes of scratch, more than its %zu",
                B, k, desc->vocab, need, kNoAllocScratchBytes);
  void* ws = nullptr;
  const int rc = accept_noalloc_scratch(&ws);
  if (rc != NJ_OK) return rc;
  hipStream_t s = (hipStream_t)stream;
  // the error word is the caller's output: it starts at zero on every call
  // (a fill kernel, not a memset, so the call can be captured in a graph)
  hipError_t e = launch_fill_i32(device_error, 0, 1, s);
  if (e != hipSuccess) return hip_fail(e, "accept_noalloc: clear error word");
  AcceptArgs a{logits, draft_tokens, draft_probs, uniforms, B, k, desc->vocab, ws, false, 0, accepted_len,
               next_tokens, device_error};
  e = launch_accept(a, s);
  return e == hipSuccess ? NJ_OK : hip_fail(e, "accept_noalloc");
}

static int gemm_args_ok(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t epilogue) {
  if (dtype != NJ_F32 && dtype != NJ_BF16) return fail(NJ_EINVAL, "bad dtype");
  if (M < 1 || N < 1 || K < 1) return fail(NJ_EINVAL, "M, N, K must be >= 1");
  if (epilogue < NJ_GEMM_STORE || epilogue > NJ_GEMM_SWIGLU) return fail(NJ_EINVAL, "bad epilogue");
  if (epilogue == NJ_GEMM_SWIGLU && N % 2) return fail(NJ_EINVAL, "SwiGLU needs an even N");
  const int Nout = epilogue == NJ_GEMM_SWIGLU ? N / 2 : N;
  if (dtype == NJ_BF16) {
    if (K % 32) return fail(NJ_EINVAL, "bf16 GEMM needs K %% 32 == 0");
    if (Nout % 16) return fail(NJ_EINVAL, "bf16 GEMM needs output width %% 16 == 0");
  }
  return NJ_OK;
}

size_t nightjar_packed_weight_elems(int32_t N, int32_t K) {
  if (N < 1 || K < 32 || K % 32) {
    fail(NJ_EINVAL, "packed weights need N >= 1 and K a positive multiple of 32");
    return 0;
  }
  return packed_weight_elems(N, K);
}

int nightjar_pack_weight(const void* src, void* dst, int32_t N, int32_t K, void* stream) {
  if (nightjar_packed_weight_elems(N, K) == 0) return NJ_EINVAL;
  if (!src || !dst) return fail(NJ_EINVAL, "NULL pointer");
  if (!aligned16(src) || !aligned16(dst)) return fail(NJ_EINVAL, "pointers must be 16-byte aligned");
  const uintptr_t s0 = (uintptr_t)src, s1 = s0 + (size_t)N * K * 2, d0 = (uintptr_t)dst,
                  d1 = d0 + packed_weight_elems(N, K) * 2;
  if (s0 < d1 && d0 < s1) return fail(NJ_EINVAL, "src and dst overlap");
  const hipError_t e = launch_pack_weight(src, dst, N, K, (hipStream_t)stream);
  return e == hipSuccess ? NJ_OK : hip_fail(e, "pack_weight");
}

size_t nightjar_gemm_workspace_bytes(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t epilogue) {
  epilogue &= ~NJ_GEMM_KBLOCKED;
  if (gemm_args_ok(dtype, M, N, K, epilogue) != NJ_OK) return 0;
  if (dtype != NJ_BF16) return kAlign;
  const GemmPlan p = gemm_plan(M, N, K, epilogue);
  return kAlign + p.counter_bytes + p.part_bytes;
}

int nightjar_gemm(int32_t dtype, const void* x, const void* w, void* y, int32_t M, int32_t N, int32_t K,
                  int32_t epilogue, void* workspace, size_t workspace_bytes, void* stream) {
  const bool kb = (epilogue & NJ_GEMM_KBLOCKED) != 0;
  epilogue &= ~NJ_GEMM_KBLOCKED;
  if (gemm_args_ok(dtype, M, N, K, epilogue) != NJ_OK) return NJ_EINVAL;
  if (kb && (dtype != NJ_BF16 || gemm_plan(M, N, K, epilogue).tile == kTileNone))
    return fail(NJ_EINVAL, "k-blocked operands need the tiled kernel");
  if (kb && epilogue == NJ_GEMM_SWIGLU && (N / 2) % 32) return fail(NJ_EINVAL, "k-blocked SwiGLU output needs F %% 32 == 0");
  if (!x || !w || !y) return fail(NJ_EINVAL, "NULL operand");
  if (dtype == NJ_BF16 && (!aligned16(x) || !aligned16(w) || !aligned16(y)))
    return fail(NJ_EINVAL, "operands must be 16-byte aligned");
  const size_t need = nightjar_gemm_workspace_bytes(dtype, M, N, K, epilogue);
  if (!workspace || workspace_bytes < need) return fail(NJ_EINVAL, "workspace NULL or smaller than %zu bytes", need);
  if (((uintptr_t)workspace & (kAlign - 1)) != 0) return fail(NJ_EINVAL, "workspace must be 256-byte aligned");
  char* ws = static_cast<char*>(workspace) + kAlign;  // [counters][partials]
  size_t cnt_bytes = 0;
  if (dtype == NJ_BF16) cnt_bytes = gemm_plan(M, N, K, epilogue).counter_bytes;
  hipError_t e = launch_gemm(dtype == NJ_BF16 ? kBF16 : kF32, x, w, y, M, N, K, epilogue, reinterpret_cast<int*>(ws),
                             reinterpret_cast<float*>(ws + cnt_bytes), (hipStream_t)stream, kb,
                             kb && epilogue == NJ_GEMM_SWIGLU);
  return e == hipSuccess ? NJ_OK : hip_fail(e, "gemm");
}

static int plan_with(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t epilogue, int32_t kernel, int32_t split,
                     GemmPlan* out) {
  if (gemm_args_ok(dtype, M, N, K, epilogue) != NJ_OK) return NJ_EINVAL;
  if (split < 0 && (kernel == NJ_GEMM_AUTO || kernel == NJ_GEMM_STREAM || kernel == NJ_GEMM_STREAM_DEEP))
    return fail(NJ_EINVAL, "split_k < 0 (stream-K) needs a tiled kernel");
  if (kernel < NJ_GEMM_AUTO || kernel > NJ_GEMM_TILE_96x128) return fail(NJ_EINVAL, "bad kernel choice");
  if (dtype != NJ_BF16) {
    if (kernel != NJ_GEMM_AUTO || split) return fail(NJ_EINVAL, "the fp32 GEMM has a single kernel and no split");
    *out = GemmPlan{};
    return NJ_OK;
  }
  if (kernel == NJ_GEMM_AUTO) {
    if (split) return fail(NJ_EINVAL, "split_k needs an explicit kernel");
    *out = gemm_plan(M, N, K, epilogue);
    return NJ_OK;
  }
  GemmPlan p;
  if (kernel == NJ_GEMM_STREAM || kernel == NJ_GEMM_STREAM_DEEP) {
    p = gemm_stream_plan(M, N, K, epilogue, split, kernel == NJ_GEMM_STREAM_DEEP ? 3 : 1);
    if (epilogue == NJ_GEMM_STORE) p = gemm_logits_widen(p, M, N);
  } else {
    if (!tile_fits(M, N, K)) return fail(NJ_EINVAL, "the tiled kernels need K %% 64 == 0 and M*K, N*K < 2^31");
    const int tile = kernel == NJ_GEMM_TILE_256x256   ? kTile256x256
                     : kernel == NJ_GEMM_TILE_192x256 ? kTile192x256
                     : kernel == NJ_GEMM_TILE_160x256 ? kTile160x256
                     : kernel == NJ_GEMM_TILE_96x256  ? kTile96x256
                     : kernel == NJ_GEMM_TILE_96x128  ? kTile96x128
                     : kernel == NJ_GEMM_TILE_128x256 ? kTile128x256
                                                      : kTile128x128;
    p = split > 0   ? gemm_tile_plan(M, N, K, epilogue, tile, std::min(split, K / 64))
        : split < 0 ? gemm_tile_plan_sk(M, N, K, epilogue, tile, -split)
                    : gemm_tile_choose(M, N, K, epilogue, tile);
  }
  if (p.nkc > 1 && p.counter_bytes > kGemmCounterBytes)
    return fail(NJ_EINVAL, "a run that splits tiles may have at most %d workgroups", kGemmMaxSplitGrid);
  if (p.tile == kTile256x256 && !tile_one_segment(p, K))
    return fail(NJ_EINVAL, "the 256x256 tile runs one tile (or one K chunk of it) per workgroup: no stream-K grid");
  if (p.part_bytes >= kMaxPartBytes) return fail(NJ_EINVAL, "split-K partials would take 2 GiB or more");
  *out = p;
  return NJ_OK;
}

size_t nightjar_gemm_plan_workspace_bytes(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t epilogue,
                                          int32_t kernel, int32_t split_k) {
  epilogue &= ~NJ_GEMM_KBLOCKED;
  GemmPlan p;
  if (plan_with(dtype, M, N, K, epilogue, kernel, split_k, &p) != NJ_OK) return 0;
  return dtype == NJ_BF16 ? kAlign + p.counter_bytes + p.part_bytes : kAlign;
}

int nightjar_gemm_with_plan(int32_t dtype, const void* x, const void* w, void* y, int32_t M, int32_t N, int32_t K,
                            int32_t epilogue, int32_t kernel, int32_t split_k, void* workspace,
                            size_t workspace_bytes, void* stream) {
  const bool kb = (epilogue & NJ_GEMM_KBLOCKED) != 0;
  epilogue &= ~NJ_GEMM_KBLOCKED;
  GemmPlan p;
  if (plan_with(dtype, M, N, K, epilogue, kernel, split_k, &p) != NJ_OK) return NJ_EINVAL;
  if (kb && (dtype != NJ_BF16 || p.tile == kTileNone)) return fail(NJ_EINVAL, "k-blocked operands need the tiled kernel");
  if (kb && epilogue == NJ_GEMM_SWIGLU && (N / 2) % 32) return fail(NJ_EINVAL, "k-blocked SwiGLU output needs F %% 32 == 0");
  if (!x || !w || !y) return fail(NJ_EINVAL, "NULL operand");
  if (dtype == NJ_BF16 && (!aligned16(x) || !aligned16(w) || !aligned16(y)))
    return fail(NJ_EINVAL, "operands must be 16-byte aligned");
  const size_t need = dtype == NJ_BF16 ? kAlign + p.counter_bytes + p.part_bytes : kAlign;
  if (!workspace || workspace_bytes < need) return fail(NJ_EINVAL, "workspace NULL or smaller than %zu bytes", need);
  if (((uintptr_t)workspace & (kAlign - 1)) != 0) return fail(NJ_EINVAL, "workspace must be 256-byte aligned");
  char* ws = static_cast<char*>(workspace) + kAlign;  // [counters][partials]
  hipError_t e;
  if (dtype == NJ_BF16)
    e = launch_gemm_plan(x, w, y, M, N, K, epilogue, p, reinterpret_cast<int*>(ws),
                         reinterpret_cast<float*>(ws + p.counter_bytes), (hipStream_t)stream, kb,
                         kb && epilogue == NJ_GEMM_SWIGLU);
  else
    e = launch_gemm(kF32, x, w, y, M, N, K, epilogue, nullptr, nullptr, (hipStream_t)stream);
  return e == hipSuccess ? NJ_OK : hip_fail(e, "gemm");
}

}  // extern "C"

namespace nj {
int set_last_error(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}
}  // namespace nj
