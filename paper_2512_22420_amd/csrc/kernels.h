// Host-side launchers of the verify-step kernels.  Each enqueues on `s` and
// returns the launch status; shapes are checked by the caller (api.cpp).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nj {

enum { kF32 = 0, kBF16 = 1 };
// kEpiLogits (internal): fp32 store plus the softmax statistics of every
// 128-wide output chunk, for the acceptance kernels.
// kEpiResidualNorm (internal): residual add that also writes the next
// RMSNorm's input (see GemmNorm).
// kEpiQkvRope (internal): QKV projection whose epilogue applies RoPE and
// stores q and the window K/V blocks (see QkvRope).
enum { kEpiStore = 0, kEpiResidual = 1, kEpiSwiglu = 2, kEpiLogits = 3, kEpiResidualNorm = 4, kEpiQkvRope = 5 };

// Output tiles of the LDS-tiled kernel for large windows: x rows x weight rows.
enum { kTileNone = 0, kTile256x256 = 1, kTile128x256 = 2, kTile128x128 = 3, kTile192x256 = 4, kTile160x256 = 5,
       kTile96x256 = 6, kTile96x128 = 7 };

// How the bf16 GEMM splits its work.  Weight-streaming kernel (tile ==
// kTileNone): 16-row x tiles per workgroup (mt), waves per workgroup (nw, 8),
// workgroups along N (ntiles) and M (mblocks).  LDS-tiled kernel: tile shape,
// ntiles / mblocks output tiles along N and M.  Both: K chunks across
// workgroups (nkc, stages_per_chunk; a stage is 256 k for the streaming kernel,
// 64 for the tiled one), and the workspace the split-K partials and arrival
// counters take.
struct GemmPlan {
  int tile;
  int mt, nw, ntiles, mblocks, nkc, stages_per_chunk;
  int depth;  // streaming kernel: weight stages in flight ahead of the one being multiplied (1 or 3)
  size_t part_bytes, counter_bytes;
  int grid;   // tiled kernel: workgroups of the stream-K schedule
  int key_m, key_n, key_k, key_epi;  // the arguments gemm_plan chose it for (its plan table checks them)
  // tiled kernel, one-segment split plans on at most kParMaxGrid workgroups:
  // every workgroup of a cut tile reduces a slice of its rows (the launch
  // also checks that the GPU has a CU for each workgroup)
  int par;
};
constexpr int kParMaxGrid = 256;
constexpr int kSplitSpinMax = 1 << 21;  // wait bound of the slice-reduced splits (~2^21 short sleeps, > 100 ms)
constexpr int kSplitErrOffset = 64;     // ints from the workspace's device-error word to a GEMM counter region
// Split-K partials through one XCD's L2 (see xcd_store): at most this many
// chunks per tile (each arrival carries a "not where round-robin dispatch put
// it" bit, bits 16 + chunk of the tile's counter).
constexpr int kSplitL2MaxChunks = 15;
// Chunks (bit c: chunk c) that act as if dispatched to a foreign XCD, for
// tests of the fallback: 0 unless NJ_TEST_SPLIT_FOREIGN is set.
unsigned split_foreign_mask();
// CUs of the current device (queried once; 0 when there is no device).
int device_cus();
// The plan the bf16 GEMM runs for y = x . w^T with epilogue epi; epi =
// kEpiQkvRope plans the QKV projection (store output), for which a
// streaming plan also applies RoPE while a tiled one needs the RoPE kernel.
// Plans of the same arguments are computed once and kept.
GemmPlan gemm_plan(int M, int N, int K, int epi);
// Plan of the LDS-tiled kernel with a given tile shape and K split (grid =
// tiles x nkc).
GemmPlan gemm_tile_plan(int M, int N, int K, int epi, int tile, int nkc);
// Plan of the LDS-tiled kernel with a given tile shape on `grid` workgroups
// that share the tiles x K/64 units of work evenly (stream-K).
GemmPlan gemm_tile_plan_sk(int M, int N, int K, int epi, int tile, int grid);
// Whether every workgroup of a tiled plan works inside one tile (grid = tiles
// x c, c <= K/64), as the 256 x 256 tile requires.
bool tile_one_segment(const GemmPlan& p, int K);
// The tiled kernel needs K % 64 == 0 and operands of fewer than 2^31 elements.
bool tile_fits(int M, int N, int K);
// Best tiled plan by the cost model (only_tile = kTileNone: any tile shape).
GemmPlan gemm_tile_choose(int M, int N, int K, int epi, int only_tile);
// Plan of the weight-streaming kernel; split > 0 forces that many K chunks
// (at most one per 256-k stage), 0 picks the split; depth 3 = three stages in
// flight per wave (1: two).
GemmPlan gemm_stream_plan(int M, int N, int K, int epi, int split, int depth);
// A streaming plan of 65..96 rows without split K, as one block of up to 6 row
// tiles for the persistent fp32-store (LM-head) kernel, which then reads the
// weights once; any other plan unchanged.  Only for plans launched through
// launch_gemm_plan / launch_gemm_logits with the store epilogue.
GemmPlan gemm_logits_widen(const GemmPlan& p, int M, int N);
int tile_bm(int tile);
int tile_bn(int tile);
// Arrival counters of split-K hand-offs live in one fixed region, whatever
// M, N, K: the streaming kernel splits K only when ntiles * mblocks <= 256,
// and a tiled run that splits tiles has at most kGemmMaxSplitGrid workgroups
// (one counter per workgroup at most).
// Arrival counters that many workgroups increment are kept 256 bytes apart:
// device-scope atomics on one cache line are serialised, so counters that
// share a line make every workgroup of a launch wait for all the others'.
constexpr int kCounterStride = 64;  // ints
constexpr int kGemmMaxSplitGrid = 1024;
constexpr size_t kGemmCounterBytes = (size_t)kGemmMaxSplitGrid * kCounterStride * 4;
// Split-K partials are addressed with 32-bit buffer offsets.
constexpr size_t kMaxPartBytes = (size_t)1 << 31;
// The planners choose no split plan whose partials exceed this, so that a
// step's partial region can be sized once for every window up to the largest
// one: windows of more than 64 rows reserve the cap, and below that the
// chosen plans' partials grow with the window.
constexpr size_t kSplitPartCap = (size_t)96 << 20;
constexpr int kTileMinRows = 65;  // windows of more than 64 rows may use the LDS-tiled kernel

// bf16 GEMM weights live in a packed layout: 128-row groups, each a run of
// K/32 k-steps of 8 tiles (16 rows x 32 k, 1 KB, MFMA lane order).  Elements
// of the packed copy of an [N][K] matrix (rows padded to a multiple of 128),
// and the kernel that writes it.
size_t packed_weight_elems(int N, int K);
hipError_t launch_pack_weight(const void* src, void* dst, int N, int K, hipStream_t s);

// y = x . w^T, x [M][K], w [N][K] (for SwiGLU N = 2F, y [M][F]); bf16 w
// packed, fp32 w row-major.  The 256 bytes before `counters` are the
// workspace's device-error word (a split GEMM whose workgroups time out
// waiting for each other sets kErrSplitWait there).  `counters`
// (plan.counter_bytes, zero on entry and on exit) and `part`
// (plan.part_bytes) are scratch; GEMMs that run one after another on a stream
// may share both as long as the counters are never overwritten by anything else.
hipError_t launch_gemm(int dtype, const void* x, const void* w, void* y, int M, int N, int K, int epi,
                       int* counters, float* part, hipStream_t s, bool x_kblocked = false, bool y_kblocked = false);
// bf16 GEMM with an explicit plan (either kernel; for the streaming one
// mt 1..4, any nkc/stages_per_chunk).
hipError_t launch_gemm_plan(const void* x, const void* w, void* y, int M, int N, int K, int epi, const GemmPlan& p,
                            int* counters, float* part, hipStream_t s, bool x_kblocked = false,
                            bool y_kblocked = false);
// LM head: y = x . w^T stored fp32, plus the chunk statistics of the
// acceptance kernels (stats [M][accept_chunks(N)][2]) when the plan uses the
// weight-streaming kernel; *stats_written says whether it did.
hipError_t launch_gemm_logits(const void* x, const void* w, float* y, float* stats, int M, int N, int K,
                              int* counters, float* part, hipStream_t s, bool* stats_written, bool x_kblocked = false);
// RMSNorm folded into the weight-streaming GEMMs.  A producer (residual
// epilogue kEpiResidualNorm) adds into h and writes xg = bf16(h * gain) and
// ssq_out[m][t], the sum of h^2 over output columns 128t .. 128t+127; a
// consumer (x = xg) scales row m of its product by
// 1 / sqrt(sum_t ssq_in[m][t] / K + eps) before its epilogue.  stats: the
// kEpiLogits chunk statistics.
struct GemmNorm {
  const float* ssq_in;  // consumer side (nullable)
  int nt_in;            // partials per row (<= 64)
  float eps;
  const void* gain;     // producer side: bf16 [N]
  void* xg;             // bf16 [M][N], or k-blocked [N/32][M][32] with xg_kb
  float* ssq_out;       // [M][ceil(N / 128)]
  float* stats;         // kEpiLogits only
  int xg_kb = 0;
};
// kEpiQkvRope: the QKV GEMM's 128-column groups are its heads (head_dim 128):
// q heads are rotated and stored to q_out [M][H][128], k heads rotated into
// the window blocks win_k [B][Hkv][16][128], v heads into win_v
// [B][Hkv][128][16]; slots T..15 of the window blocks are zeroed.  Rotate-half
// pairs (j, j+64) turn by the step's RoPE table cs [M][64] of (cos, sin)
// (written by launch_embed_gather).  Workgroup 0 also stores ctx_snap
// (nullable) and clears the attention split counters attn_cnt [B*Hkv]
// (nullable).
struct QkvRope {
  const int32_t* ctx;
  int T, H, Hkv;
  const float* cs;
  void* q_out;
  void* win_k;
  void* win_v;
  int32_t* ctx_snap;
  int* attn_cnt;
};
// Whether gemm_plan picks the weight-streaming kernel for this shape (the
// only one with the folded norm).
bool gemm_streams(int M, int N, int K, int epi);
// (max, sum of exp) pairs per row that the LM-head GEMM's statistics epilogue
// writes: one per 128-column chunk, per persistent workgroup, or per column tile
int logits_stat_entries(int M, int N, int K);
// A tiled plan takes the row scale in any epilogue and the next norm's inputs
// only from a slice-reduced residual plan (not QKV + RoPE); x_kblocked: x is
// k-blocked (tiled plans only); y_kblocked: the SwiGLU output k-blocked.
hipError_t launch_gemm_norm(const void* x, const void* w, void* y, int M, int N, int K, int epi, const GemmNorm& nm,
                            int* counters, float* part, hipStream_t s, const QkvRope* rope = nullptr,
                            bool x_kblocked = false, bool y_kblocked = false);
// The LDS-tiled kernel alone (K % 64 == 0).  x_kblocked: x is stored
// k-blocked, [K/32][M][32] (element (m, k) at ((k / 32) * M + m) * 32 + k % 32),
// so that each 16-row x 32-column operand unit is 1 KB of contiguous memory;
// y_kblocked: the SwiGLU output [M][F] is written that way too (as the next
// tiled GEMM's input).
hipError_t launch_gemm_tile(const void* x, const void* w, void* y, int M, int N, int K, int epi, const GemmPlan& p,
                            int* counters, float* part, hipStream_t s,
                            float* stats = nullptr, bool x_kblocked = false, bool y_kblocked = false,
                            const GemmNorm* nm = nullptr);

// h[r] = E[id(r)], x[r] = rmsnorm(h[r]) * gain, ids from last/draft tokens.
struct AttnPlan;
// The embedding kernels can carry one more workgroup that builds the
// attention's work list (plan nullable; see attn_work.h).
// With rope_cs (bf16, 128-dim heads) it also writes the step's RoPE table, as
// launch_embed_gather does, for a QKV GEMM with the RoPE epilogue.
hipError_t launch_embed_norm(int dtype, const int32_t* last, const int32_t* drafts, int B, int T,
                             const void* embed, const void* gain, float* h, void* x, int d, int V,
                             float eps, int* err, hipStream_t s, bool x_kblocked = false,
                             const AttnPlan* plan = nullptr, const int32_t* ctx = nullptr, float theta = 0.f,
                             float* rope_cs = nullptr);

// bf16, norm folded into the GEMMs: h[r] = E[id(r)], x[r] = bf16(h[r] * gain),
// ssq[r][t] = sum of h[r]^2 over columns 128t .. 128t+127; and the step's RoPE
// table rope_cs[r][j] = (cos, sin) of (ctx[b] + i) * theta^(-j/64) (nullable).
hipError_t launch_embed_gather(const int32_t* last, const int32_t* drafts, int B, int T, const void* embed,
                               const void* gain, float* h, void* x, float* ssq, int d, int V, int* err,
                               const int32_t* ctx, float theta, float* rope_cs, hipStream_t s,
                               const AttnPlan* plan = nullptr);

// The same outputs (x, ssq, rope_cs) for given residual rows h [B*T][d] fp32
// instead of embedding rows (h is only read).
hipError_t launch_norm_inputs(const float* h, int B, int T, const void* gain, void* x, float* ssq, int d,
                              const int32_t* ctx, float theta, float* rope_cs, hipStream_t s);

// x[r] = rmsnorm(h[r]) * gain; x row-major, or k-blocked (as launch_gemm_tile reads it)
hipError_t launch_rmsnorm(int dtype, const float* h, const void* gain, void* x, int M, int d, float eps,
                          hipStream_t s, bool x_kblocked = false);

// RoPE on q and k rows of qkv at positions ctx[b] + i; q -> q_out [M][H][D];
// k, v -> one 16-slot window block per (b, kv head).  D <= 2 * kMaxHalfDim.
constexpr int kMaxHalfDim = 256;
struct RopeFreq {
  double inv_freq[kMaxHalfDim];  // theta^(-2j/D)
};
// ctx_snap (nullable): receives ctx[b], the positions the KV append uses.
// attn_counters (nullable): [B*Hkv] cleared for the attention launch that follows.
hipError_t launch_rope_window(int dtype, const float* qkv, const int32_t* ctx, int B, int T, int H, int Hkv,
                              int D, float theta, void* q_out, void* win_k, void* win_v, int32_t* ctx_snap,
                              int* attn_counters, hipStream_t s);

struct AttnWork;
struct AttnArgs {
  int dtype;
  const void* q;        // [M][H][D]
  const void* k_pages;  // [nb][Hkv][16][D]
  const void* v_pages;  // [nb][Hkv][D][16]
  const void* win_k;    // [B][Hkv][16][D]
  const void* win_v;    // [B][Hkv][D][16]
  const int32_t* block_table;
  int max_blocks;
  const int32_t* ctx;
  int num_blocks, B, T, H, Hkv, D;
  float* part_o;        // split partials (bf16 path)
  float* part_ml;
  int* counters;         // [B*Hkv] split arrivals, zero on entry (bf16 path)
  int wgs;              // bf16: workgroups of the attention work list (attention_plan)
  const AttnWork* work; // bf16: the list, built by launch_attn_plan or the embedding kernel
  void* out;            // [M][H*D]; k-blocked [H*D/32][M][32] when out_kblocked (bf16 path)
  int* err;
  bool out_kblocked;
};
// Workgroups of the bf16 path's work list, the bytes of the list, and the
// partial buffer floats the splits need.
int attention_plan(int B, int Hkv, int max_blocks);
// Whether a work list of nwg workgroups is ordered longest split first: when
// the grid is more than one round of resident attention workgroups.
bool attention_orders(int nwg);
size_t attention_work_bytes(int B, int Hkv);
size_t attention_partial_floats(int B, int Hkv, int T, int G, int D);
// The work list for attention launches over these context lengths (one
// workgroup), clearing their split counters when `counters` is given.
hipError_t launch_attn_plan(const int32_t* ctx, int B, int Hkv, int T, int max_blocks, int nwg, void* work,
                            int* counters, hipStream_t s);
hipError_t launch_attention(const AttnArgs& a, hipStream_t s);

// Acceptance from logits [B*T][V].
struct AcceptArgs {
  const float* logits;
  const int32_t* drafts;    // [B][k]
  const float* dprobs;      // [B][k][V]
  const float* uniforms;    // [B][k+1]
  int B, k, V;
  void* scratch;            // accept_workspace_bytes(B*T, V) bytes
  bool stats_ready;         // the chunk statistics at accept_stats_ptr(scratch) are already written
  int stat_entries;         // stats_ready: (max, sum) pairs per row written (row stride accept_chunks(V))
  int32_t* accepted_len;
  int32_t* next_tokens;
  int* err;
};
int accept_chunks(int V);
float* accept_stats_ptr(void* scratch);  // [B*T][accept_chunks(V)][2] chunk max, sum of exp
size_t accept_workspace_bytes(int rows, int V);
hipError_t launch_accept(const AcceptArgs& a, hipStream_t s);
// After launch_accept of a k = 0 step: the drawn tokens to tokens[b * tstride]
// and the distributions p = softmax(logits row) to probs[b * pstride ...].
hipError_t launch_emit_draft(const AcceptArgs& a, int32_t* tokens, int tstride, float* probs, long long pstride,
                             hipStream_t s);

struct KvAppendArgs {
  int dtype;
  void* const* k_pages;      // host array of L device pointers
  void* const* v_pages;
  const void* win_k;         // [L][B][Hkv][16][D]
  const void* win_v;         // [L][B][Hkv][D][16]
  const int32_t* block_table;
  int max_blocks, num_blocks;
  const int32_t* ctx_snap;   // [B] context lengths the verify step read
  int32_t* ctx;              // [B] set to ctx_snap + n + 1
  const int32_t* accepted_len;
  int L, B, k, Hkv, D;       // D % 8 == 0
  int* err;
};
hipError_t launch_kv_append(const KvAppendArgs& a, hipStream_t s);

hipError_t launch_fill_i32(int32_t* p, int32_t v, int n, hipStream_t s);
hipError_t launch_copy_i32(int32_t* dst, const int32_t* src, int n, hipStream_t s);
// dst[i] = src[i * stride] for 32-bit words, i < n.
hipError_t launch_gather_u32(int32_t* dst, const int32_t* src, int n, int stride, hipStream_t s);

// Sets the message nightjar_last_error() returns on this thread; returns code.
int set_last_error(int code, const char* fmt, ...);

}  // namespace nj
