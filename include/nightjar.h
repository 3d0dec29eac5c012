/*
 * nightjar.h -- C ABI of the batched speculative verify step on MI355X (gfx950).
 *
 * Nightjar (arXiv 2512.22420) serves requests with speculative decoding whose
 * speculative length gamma is chosen per batch size B by a bandit planner
 * (Sec. 5), gamma = 0 meaning plain decoding (Sec. 4).  The computation whose
 * cost that planner trades off is the verify step: the target model scores
 * all gamma drafts of each of the B sequences in one forward pass (Sec. 2.2),
 * the acceptance test keeps the longest accepted prefix and adds one corrected
 * or bonus token (Sec. 3.1; Sec. 5.1 "committed tokens"), and only accepted
 * tokens' keys and values are committed to the paged KV cache before the next
 * step (PagedAttention, Sec. 2.1; step-level finalisation, Sec. 6.5).
 *
 * In this header gamma is written k.  The target is a Llama-style decoder:
 * RMSNorm, rotate-half RoPE, grouped-query attention, SwiGLU FFN, untied LM
 * head, no biases.
 *
 * Conventions for every entry point
 * ---------------------------------
 * - Pointers marked "device" are device memory on the current HIP device and
 *   stay owned by the caller; descriptor structs and pointer arrays inside them
 *   are host memory, read during the call only.
 * - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *   stream) and makes no device allocation; scratch lives in the caller's
 *   workspace.
 * - Return value: NJ_OK (0) on success, otherwise a negative NJ_E* code and
 *   nightjar_last_error() describes the problem.  Argument errors are found on
 *   the host before anything is enqueued.  Bad data found by the kernels (token
 *   or block ids out of range, a context that does not fit the block table)
 *   is skipped without any out-of-bounds access and recorded in the workspace;
 *   nightjar_device_error() reports it.  Outputs are undefined after an error.
 * - Element types: dtype NJ_BF16 stores weights, KV pages and window K/V as
 *   bf16 (round-to-nearest-even); NJ_F32 stores them as fp32.  Logits,
 *   draft probabilities and uniforms are fp32 in both; ids are int32.
 *
 * Layouts (row-major, reduction dimension contiguous)
 * ----------------------------------------------------
 *   embed, lm_head     [V][d]
 *   w_qkv              [(H + 2*Hkv) * D][d]   query rows, then key rows, then value rows
 *   w_o                [d][H * D]
 *   w_gate_up          [2F][d]                gate rows, then up rows
 *   w_down             [d][F]
 *   norms              [d]
 *   k_pages[l]         [num_blocks][Hkv][block_size][D]
 *   v_pages[l]         [num_blocks][Hkv][D][block_size]   (dim-major inside a block)
 *   block_table        [B][max_blocks]   logical block j of sequence b -> physical block
 *   Cached K is stored after RoPE; V as is.  Token t of sequence b lives in
 *   block block_table[b][t / block_size], slot t % block_size.  block_size
 *   must be 16.
 */
#ifndef NIGHTJAR_H
#define NIGHTJAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { NJ_F32 = 0, NJ_BF16 = 1 };

enum {
  NJ_OK = 0,
  NJ_EINVAL = -1,  /* bad argument (null pointer, bad size, workspace too small, ...) */
  NJ_EDEVICE = -2, /* the kernels found bad data (see nightjar_device_error)          */
  NJ_EHIP = -3     /* a HIP runtime call failed                                       */
};

/* Device-side error bits reported by nightjar_device_error(). */
enum {
  NJ_DEV_BAD_TOKEN = 1,   /* a window or draft token id outside [0, V)                 */
  NJ_DEV_BAD_BLOCK = 2,   /* a needed block-table entry outside [0, num_blocks)          */
  NJ_DEV_BAD_CONTEXT = 4, /* context_lens[b] < 0 or context_lens[b]+k+1 > max_blocks*16  */
  NJ_DEV_BAD_ACCEPT = 8,  /* kv_append: accepted_len[b] outside [0, k]                   */
  NJ_DEV_SPLIT_WAIT = 16  /* a split GEMM's workgroups did not all arrive within the wait
                             bound (the GPU ran fewer of them at once than the plan
                             assumes); the GEMM's output is not valid                     */
};

typedef struct nj_model_desc {
  int32_t n_layers;   /* L                      */
  int32_t d_model;    /* d                      */
  int32_t n_heads;    /* H query heads          */
  int32_t n_kv_heads; /* Hkv; H % Hkv == 0      */
  int32_t head_dim;   /* D (multiple of 8)      */
  int32_t ffn_dim;    /* F                      */
  int32_t vocab;      /* V                      */
  int32_t block_size; /* tokens per KV block: 16 */
  float rms_eps;
  float rope_theta;
  int32_t dtype;      /* NJ_F32 or NJ_BF16      */
} nj_model_desc;

/*
 * Weight matrices (w_qkv, w_o, w_gate_up, w_down, lm_head) are [N][K] with
 * y = x . w^T.  fp32 models pass them row-major.  bf16 models pass them in
 * the packed layout written by nightjar_pack_weight (see there); the
 * embedding and the norm gains are always plain arrays.
 */
typedef struct nj_layer_weights {
  const void* attn_norm; /* [d]                    */
  const void* w_qkv;     /* [(H+2Hkv)*D][d]        */
  const void* w_o;       /* [d][H*D]               */
  const void* ffn_norm;  /* [d]                    */
  const void* w_gate_up; /* [2F][d]: gate rows, then up rows */
  const void* w_down;    /* [d][F]                 */
} nj_layer_weights;

typedef struct nj_weights {
  const void* embed;              /* device [V][d] row-major            */
  const void* final_norm;         /* device [d]                         */
  const void* lm_head;            /* device [V][d]                      */
  const nj_layer_weights* layers; /* host array of n_layers; entries are device pointers */
} nj_weights;

typedef struct nj_kv_cache {
  void* const* k_pages; /* host array of n_layers device pointers: [num_blocks][Hkv][16][D] */
  void* const* v_pages; /* host array of n_layers device pointers: [num_blocks][Hkv][D][16] */
  int32_t num_blocks;
} nj_kv_cache;

/*
 * Bytes of workspace a verify step with up to max_B sequences and up to max_k
 * drafts each needs (0 if the descriptor is invalid).  A workspace sized for
 * (max_B, max_k) serves every smaller (B, k).
 */
size_t nightjar_workspace_bytes(const nj_model_desc* desc, int32_t max_B, int32_t max_k);

/*
 * Whether a verify step of B sequences with k drafts folds its RMSNorms into
 * the neighbouring GEMMs (1) or runs them as their own kernels (0); < 0 on bad
 * arguments.  The two differ only in where bf16 rounding happens: folded, a
 * GEMM input is bf16(h * gain) and the 1/rms row scale is applied to the fp32
 * product; unfused, the input is bf16(RMSNorm(h) * gain).  Windows of up to
 * ~64 rows (bf16, every GEMM on the weight-streaming kernel) fold.
 */
int nightjar_step_folds_norms(const nj_model_desc* desc, int32_t B, int32_t k);

/*
 * Prepare a fresh workspace: zero-fills it (the device error word and the
 * split-K arrival counters must start at zero).  Call once after allocating
 * it; device memory, 256-byte aligned.
 */
int nightjar_workspace_init(void* workspace, size_t workspace_bytes, void* stream);

/*
 * nightjar_verify_step -- one speculative verify step for B sequences with k
 * drafts each (Sec. 2.2 "verifying": all k drafts scored in one target forward;
 * Sec. 3.1: n accepted plus one token committed).
 *
 * Window of sequence b: token 0 is last_tokens[b] (the last committed token,
 * whose KV is not yet cached), tokens 1..k are draft_tokens[b][0..k-1]; window
 * token i sits at position context_lens[b] + i and attends to every cached
 * token of b and to window tokens 0..i.  Target row i gives p_i, the target
 * distribution of the token after window token i (softmax of the logits,
 * temperature 1, no truncation).
 *
 * Acceptance (the standard speculative-sampling test the paper cites; its
 * output distribution is the target's, Sec. 1 and Sec. 6.5): for i = 0..k-1,
 * draft x = draft_tokens[b][i] is accepted iff uniforms[b][i] < p_i(x) / q_i(x)
 * with q_i(x) = draft_probs[b][i][x] (q_i(x) == 0 counts as accepted); the
 * first rejection at n stops the loop and one token is drawn from
 * max(0, p_n - q_n) (from p_n if that is all zero); if all k are accepted the
 * bonus token is drawn from p_k.  The draw uses uniforms[b][k]: the smallest j
 * whose running sum of weights (index order) exceeds uniforms[b][k] times the
 * total.
 *
 *   desc, w, kv         model and cache (see layouts above)
 *   block_table         device int32 [B][max_blocks]
 *   context_lens        device int32 [B]   cached tokens per sequence (not modified)
 *   last_tokens         device int32 [B]
 *   draft_tokens        device int32 [B][k]      may be NULL when k == 0
 *   draft_probs         device fp32  [B][k][V]   may be NULL when k == 0
 *   uniforms            device fp32  [B][k+1]    values in [0, 1)
 *   B >= 1, 0 <= k <= 15 (the window fits one 16-token block)
 *   accepted_len        device int32 [B]         out: n_b
 *   next_tokens         device int32 [B][k+1]    out: drafts[0..n_b-1], the drawn token, then -1
 *   target_logits       device fp32  [B][k+1][V] out, or NULL (then kept in the workspace)
 *   workspace           device, >= nightjar_workspace_bytes(desc, B, k) bytes; it also
 *                       keeps the window K/V for the following nightjar_kv_append
 */
int nightjar_verify_step(const nj_model_desc* desc, const nj_weights* w, const nj_kv_cache* kv,
                         const int32_t* block_table, int32_t max_blocks, const int32_t* context_lens,
                         const int32_t* last_tokens, const int32_t* draft_tokens, const float* draft_probs,
                         const float* uniforms, int32_t B, int32_t k,
                         int32_t* accepted_len, int32_t* next_tokens, float* target_logits,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * nightjar_draft_step -- one token of the draft model's chain (Sec. 2.2: a
 * small draft model proposes the k tokens one at a time).  The draft model is
 * a decoder of the same family (descriptor, weights and paged cache as for the
 * target); this is a k = 0 verify step on it: a forward of last_tokens[b] at
 * position context_lens[b], the token drawn from its distribution p (softmax
 * of the logits) with uniforms[b], and p itself recorded as the draft
 * distribution q that the target's acceptance test divides by.
 *
 *   last_tokens   device int32 [B]; uniforms device fp32 [B] in [0, 1)
 *   token_out     device int32: token of sequence b at token_out[b * token_stride]
 *   probs_out     device fp32: p of sequence b at probs_out[b * probs_stride + j],
 *                 j < vocab (probs_stride >= vocab); with strides k and k*V the
 *                 outputs of chain position i fill column i of the target's
 *                 draft_tokens [B][k] and draft_probs [B][k][V]
 *   workspace     as for nightjar_verify_step with (B, 0); a following
 *                 nightjar_kv_append with k = 0 commits the input token's KV
 */
int nightjar_draft_step(const nj_model_desc* desc, const nj_weights* w, const nj_kv_cache* kv,
                        const int32_t* block_table, int32_t max_blocks, const int32_t* context_lens,
                        const int32_t* last_tokens, const float* uniforms, int32_t B, int32_t* token_out,
                        int32_t token_stride, float* probs_out, int64_t probs_stride, void* workspace,
                        size_t workspace_bytes, void* stream);

/*
 * nightjar_sd_step -- one whole speculative-decoding step (Sec. 2.2, Sec. 3.1:
 * the draft proposes k tokens, the target verifies them in one forward, n
 * accepted plus one token are committed; k = 0 is plain decoding, Sec. 4).
 * The draft and target caches share one block table and one context-length
 * array (a logical block holds the same 16 positions in both pools) and must
 * be in step when k > 0.  For k > 0: k+1 draft forwards (forward i reads the
 * previous token and draws draft i+1 with draft_uniforms[b][i]; forward k only
 * commits draft k's KV, its draw is discarded), each followed by the draft's
 * KV append; then the target's verify step and KV append.  After the step the
 * draft cache holds the same committed tokens as the target's (positions past
 * context_lens are ignored).  With k = 0 the draft does not run and its cache
 * falls behind: re-enabling speculation then needs the draft KV rebuilt (the
 * switching cost the planner accounts for, Sec. 5.2), which is the caller's.
 *
 *   context_lens     device int32 [B], in/out (advanced by accepted_len + 1)
 *   draft_uniforms   device fp32 [B][k+1]; uniforms device fp32 [B][k+1] (the target's)
 *   draft_tokens     device int32 [B][k], out; draft_probs device fp32 [B][k][V], out
 *   accepted_len, next_tokens: out, as for nightjar_verify_step
 *   target_ws        >= nightjar_workspace_bytes(target, B, k)
 *   draft_ws         >= nightjar_sd_workspace_bytes(draft, B); both zero-filled once
 */
size_t nightjar_sd_workspace_bytes(const nj_model_desc* draft, int32_t B);
int nightjar_sd_step(const nj_model_desc* target, const nj_weights* tw, const nj_kv_cache* tkv,
                     const nj_model_desc* draft, const nj_weights* dw, const nj_kv_cache* dkv,
                     const int32_t* block_table, int32_t max_blocks, int32_t* context_lens,
                     const int32_t* last_tokens, const float* draft_uniforms, const float* uniforms, int32_t B,
                     int32_t k, int32_t* draft_tokens, float* draft_probs, int32_t* accepted_len,
                     int32_t* next_tokens, void* target_ws, size_t target_ws_bytes, void* draft_ws,
                     size_t draft_ws_bytes, void* stream);

/*
 * nightjar_kv_append -- commit the accepted window rows (Sec. 6.5: a step is
 * finalised before the next begins; rejected drafts leave no KV behind).
 *
 * For each b, window rows 0..accepted_len[b] (the last committed token plus the
 * accepted drafts) are written to positions c_b + j of the pages, where c_b is
 * context_lens[b] as the verify step read it (the positions its RoPE used,
 * kept in the workspace), then context_lens[b] = c_b + accepted_len[b] + 1 on
 * the device.  The emitted token is not appended: it is the next step's last
 * token.  Must follow the nightjar_verify_step that filled `workspace`, with
 * the same desc, kv, block_table, max_blocks, B and k, before another verify
 * step reuses it.  Page arrays must be 16-byte aligned.
 *
 *   context_lens   device int32 [B], out (overwritten as above)
 *   accepted_len   device int32 [B]
 */
int nightjar_kv_append(const nj_model_desc* desc, const nj_kv_cache* kv, const int32_t* block_table,
                       int32_t max_blocks, int32_t* context_lens, const int32_t* accepted_len,
                       int32_t B, int32_t k, const void* workspace, size_t workspace_bytes, void* stream);

/*
 * Waits for `stream`, then returns the NJ_DEV_* bits the kernels recorded in
 * `workspace` since the last call (and clears them), or a negative NJ_E* code.
 */
int nightjar_device_error(void* workspace, size_t workspace_bytes, void* stream);

/* Message of the last failed call on this thread ("" if none). */
const char* nightjar_last_error(void);

/* ---------------------------------------------------------------------------
 * Kernel timing of the verify step, for benchmarks: while enabled, every
 * launch site of nightjar_verify_step and nightjar_kv_append records a pair of
 * HIP events around its kernels on the call's stream (a little host work and
 * two event records per launch site; not for use under graph capture).
 * nightjar_profile_read waits for the recorded events and returns the mean
 * time per launch of one kernel class since the last nightjar_profile_enable.
 * ------------------------------------------------------------------------- */
enum {
  NJ_PROF_EMBED = 0,     /* token assembly, embedding gather, first norm inputs, RoPE table */
  NJ_PROF_QKV = 1,       /* QKV GEMM (with its RoPE and window store when the norm is folded) */
  NJ_PROF_NORM = 2,      /* stand-alone RMSNorm kernels (windows whose norms are not folded) */
  NJ_PROF_ROPE = 3,      /* stand-alone RoPE + window K/V store (idem)                        */
  NJ_PROF_ATTENTION = 4, /* paged verify attention (with its split merge)                     */
  NJ_PROF_O = 5,         /* O GEMM + residual                                                 */
  NJ_PROF_GATE_UP = 6,   /* gate/up GEMM + SwiGLU                                             */
  NJ_PROF_DOWN = 7,      /* down GEMM + residual                                              */
  NJ_PROF_LM_HEAD = 8,   /* final norm (folded) + LM head + softmax statistics                */
  NJ_PROF_ACCEPT = 9,    /* acceptance (2 or 3 kernels)                                       */
  NJ_PROF_KV_APPEND = 10,
  NJ_PROF_COUNT = 11
};
int nightjar_profile_enable(int32_t enable); /* also resets the totals */
int nightjar_profile_read(int32_t kernel, double* mean_us, int64_t* launches);

/* ---------------------------------------------------------------------------
 * Stage entry points: single stages of the verify step, with the kernels the
 * step uses, for stage-level parity tests and kernel timing.
 * ------------------------------------------------------------------------- */

/*
 * Acceptance alone, from given target logits (the acceptance rule above).
 *   logits [B][k+1][V] fp32, draft_tokens [B][k], draft_probs [B][k][V],
 *   uniforms [B][k+1]; outputs as in nightjar_verify_step.  Only desc->vocab
 *   is read.  workspace: device, 256-byte aligned, at least
 *   nightjar_accept_workspace_bytes(vocab, B, k) bytes, zero-filled once by
 *   nightjar_workspace_init.
 */
size_t nightjar_accept_workspace_bytes(int32_t vocab, int32_t B, int32_t k);
int nightjar_accept(const nj_model_desc* desc, const float* logits, const int32_t* draft_tokens,
                    const float* draft_probs, const float* uniforms, int32_t B, int32_t k,
                    int32_t* accepted_len, int32_t* next_tokens, void* workspace, size_t workspace_bytes,
                    void* stream);

/*
 * nightjar_rmsnorm_rope -- the inputs of one layer's attention (a stage of the
 * verify step, with the kernels the step uses for a window of B*(k+1) rows):
 * x = RMSNorm(h) * attn_norm (x / sqrt(mean(x^2) + eps), the Llama-style
 * decoder's pre-attention norm), [q | k | v] = x . w_qkv^T, then rotate-half
 * RoPE on q and k at position context_lens[b] + i for window row i of
 * sequence b (pair (j, j + D/2) turns by pos * rope_theta^(-2j/D)).  Window K
 * and V go to one 16-slot block per (sequence, KV head), in the layout of a
 * page block, ready for nightjar_attn_verify (Sec. 2.2: all drafts are scored
 * in one forward; Sec. 2.1: paged K/V blocks).
 *
 *   h             device fp32 [B*(k+1)][d]   residual rows (row b*(k+1)+i)
 *   attn_norm     device [d] (desc dtype)
 *   w_qkv         device [(H+2Hkv)*D][d]: bf16 packed (nightjar_pack_weight), fp32 row-major
 *   context_lens  device int32 [B]
 *   q_out         device [B*(k+1)][H][D] (desc dtype), rotated queries
 *   win_k         device [B][Hkv][16][D]: rotated keys in slots 0..k, slots k+1..15 zero
 *   win_v         device [B][Hkv][D][16]: values in slots 0..k, slots k+1..15 zero
 *   workspace     device, 256-byte aligned, >= nightjar_rmsnorm_rope_workspace_bytes(desc, B, k),
 *                 zero-filled once by nightjar_workspace_init
 * Every pointer 16-byte aligned.  Only the descriptor's d_model, heads,
 * head_dim, rms_eps, rope_theta and dtype are used (plus ffn_dim and vocab,
 * which decide, as in the step, whether the norm is folded into the GEMM).
 */
size_t nightjar_rmsnorm_rope_workspace_bytes(const nj_model_desc* desc, int32_t B, int32_t k);
int nightjar_rmsnorm_rope(const nj_model_desc* desc, const float* h, const void* attn_norm, const void* w_qkv,
                          const int32_t* context_lens, int32_t B, int32_t k, void* q_out, void* win_k, void* win_v,
                          void* workspace, size_t workspace_bytes, void* stream);

/*
 * nightjar_attn_verify -- paged verify attention of one layer (Sec. 2.1:
 * PagedAttention, cached K/V in 16-token blocks reached through a block table;
 * Sec. 2.2: the k+1 window tokens of each sequence are scored together).
 * Window query i of sequence b attends to the context_lens[b] cached tokens of
 * b and to window tokens 0..i; query head h reads KV head h / (H / Hkv);
 * scores q.k / sqrt(D), softmax, weighted sum of values.
 *
 *   q              device [B*(k+1)][H][D] (desc dtype)
 *   k_pages        device [num_blocks][Hkv][16][D]    one layer's pages
 *   v_pages        device [num_blocks][Hkv][D][16]
 *   win_k, win_v   device, the window blocks as nightjar_rmsnorm_rope writes them
 *   block_table    device int32 [B][max_blocks]; context_lens device int32 [B]
 *   out            device [B*(k+1)][H*D] (desc dtype)
 *   workspace      device, 256-byte aligned, >= nightjar_attn_workspace_bytes(desc, B, k),
 *                  zero-filled once by nightjar_workspace_init; device errors
 *                  (NJ_DEV_BAD_BLOCK, NJ_DEV_BAD_CONTEXT) are read from it with
 *                  nightjar_device_error
 * bf16: (k+1) * (H/Hkv) <= 64 and 16-byte aligned pointers; fp32: max_blocks <= 1024.
 */
size_t nightjar_attn_workspace_bytes(const nj_model_desc* desc, int32_t B, int32_t k);
int nightjar_attn_verify(const nj_model_desc* desc, const void* q, const void* k_pages, const void* v_pages,
                         int32_t num_blocks, const void* win_k, const void* win_v, const int32_t* block_table,
                         int32_t max_blocks, const int32_t* context_lens, int32_t B, int32_t k, void* out,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * nightjar_accept_noalloc -- nightjar_accept with no workspace, for callers
 * that cannot allocate device memory (code under HIP graph capture, serving
 * loops and harnesses that forbid hipMalloc).  Same rule, same kernels, same
 * outputs bit for bit as nightjar_accept.  Its scratch is a fixed array of
 * 32 MiB of device memory, one per GPU, that the library holds until the
 * process ends; a call whose
 * B * (k+1) rows and vocabulary need more (about rows * vocab * 3/32 bytes)
 * fails with NJ_EINVAL before anything is enqueued.  The call allocates
 * nothing (its first call on a device looks up that device's copy of the
 * array).  Every call on one GPU shares that GPU's array: calls that overlap
 * in time on one GPU (other streams, other threads) race and give undefined
 * outputs; calls in order on one stream are safe.
 *
 *   device_error   device int32, out: the NJ_DEV_* bits this call found (0 if none);
 *                  read it after the stream has finished
 * The other arguments as in nightjar_accept.
 */
int nightjar_accept_noalloc(const nj_model_desc* desc, const float* logits, const int32_t* draft_tokens,
                            const float* draft_probs, const float* uniforms, int32_t B, int32_t k,
                            int32_t* accepted_len, int32_t* next_tokens, int32_t* device_error, void* stream);

/*
 * Packed layout of a bf16 weight matrix w [N][K] (K % 32 == 0), the form in
 * which the bf16 GEMMs read their weights (a layout choice of this library,
 * not of the method: every load instruction of the GEMM kernels reads 1 KB of
 * contiguous memory).  Rows are taken in groups of 128 (the last group padded
 * with zero rows); a group is K/32 consecutive k-steps; a k-step is 8 tiles of
 * 16 rows x 32 k; a tile is 1 KB, element (r, c) of the tile at position
 * ((c / 8) * 16 + r) * 8 + c % 8.  So element (n, k) lands at
 *   ((((n / 128) * (K / 32) + k / 32) * 8 + (n / 16) % 8) * 64
 *     + ((k % 32) / 8) * 16 + n % 16) * 8 + k % 8.
 * nightjar_packed_weight_elems returns the element count of the packed copy
 * (0 for bad sizes); nightjar_pack_weight writes it (src row-major [N][K],
 * dst of packed_weight_elems elements, both device memory, 16-byte aligned,
 * not overlapping), asynchronously on `stream`.  Returns NJ_OK, NJ_EINVAL
 * (bad sizes, NULL or misaligned pointers) or NJ_EHIP.
 */
size_t nightjar_packed_weight_elems(int32_t N, int32_t K);
int nightjar_pack_weight(const void* src, void* dst, int32_t N, int32_t K, void* stream);

/* Epilogues of nightjar_gemm. */
enum {
  NJ_GEMM_STORE = 0,    /* y[m][n] = acc (fp32 out)                                  */
  NJ_GEMM_RESIDUAL = 1, /* y[m][n] += acc (fp32 in/out)                              */
  NJ_GEMM_SWIGLU = 2,   /* N = 2F weight rows; y[m][f] = silu(acc_f) * acc_{F+f}, y in
                           the weight dtype, [M][F]                                 */
  /* Flag OR-ed into the epilogue: x (and a SWIGLU y) in the k-blocked layout
     the verify step gives the tiled kernel's inputs, [K/32][M][32]: element
     (m, k) at ((k / 32) * M + m) * 32 + k % 32 (for y, F in place of K; F % 32
     == 0).  bf16 and the tiled kernel only (nightjar_gemm: when its planner picks that
     kernel); otherwise NJ_EINVAL. */
  NJ_GEMM_KBLOCKED = 16
};

/*
 * y = x . w^T with the step's GEMM kernels.  x [M][K] and w [N][K] in `dtype`
 * (NJ_BF16 or NJ_F32), device, 16-byte aligned, a bf16 w in the packed layout
 * of nightjar_pack_weight; y as the epilogue says.
 * M >= 1; for bf16 K % 32 == 0 and the output width % 16 == 0.  workspace:
 * device, 256-byte aligned, at least nightjar_gemm_workspace_bytes(...) bytes,
 * prepared once with nightjar_workspace_init (split-K counters start at zero
 * and are left at zero by every call).
 */
size_t nightjar_gemm_workspace_bytes(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t epilogue);
int nightjar_gemm(int32_t dtype, const void* x, const void* w, void* y, int32_t M, int32_t N, int32_t K,
                  int32_t epilogue, void* workspace, size_t workspace_bytes, void* stream);

/* Kernel choices of nightjar_gemm_with_plan. */
enum {
  NJ_GEMM_AUTO = 0,         /* the kernel and split nightjar_gemm picks              */
  NJ_GEMM_STREAM = 1,       /* weight-streaming kernel (windows up to ~128 rows)     */
  NJ_GEMM_TILE_256x256 = 2, /* LDS-tiled kernel; output tile = x rows x weight rows  */
  NJ_GEMM_TILE_128x256 = 3,
  NJ_GEMM_TILE_128x128 = 4,
  NJ_GEMM_STREAM_DEEP = 5,  /* weight-streaming kernel, 3 stages in flight per wave  */
  NJ_GEMM_TILE_192x256 = 6, /* LDS-tiled kernel, 192-row x tiles (windows of 3 x 64 rows)    */
  NJ_GEMM_TILE_160x256 = 7, /* LDS-tiled kernel, 160-row x tiles (windows of 2 x 160 rows)   */
  NJ_GEMM_TILE_96x256 = 8,  /* LDS-tiled kernels with small tiles, for weight matrices      */
  NJ_GEMM_TILE_96x128 = 9   /* with few rows (more tiles to fill the chip)                  */
};

/*
 * nightjar_gemm with the kernel and the number of K chunks chosen by the
 * caller, for parity tests of every kernel shape and for tuning.  split_k = 0
 * lets the kernel's planner choose; split_k >= 1 is capped so that every chunk
 * has work (128 k per chunk at least for NJ_GEMM_STREAM, 64 for the tiled
 * kernels).  For the tiled kernels split_k = -G runs G workgroups that share
 * the output tiles x K/64 units of work evenly (stream-K; G capped at the unit
 * count), tiles cut between workgroups being summed in k order.  The tiled
 * kernels need K % 64 == 0, and a run that cuts tiles may have at most 1024
 * workgroups; otherwise NJ_EINVAL.  Operands, epilogues and errors
 * as in nightjar_gemm; the workspace must hold
 * nightjar_gemm_plan_workspace_bytes(...) bytes (0 = invalid arguments).
 */
size_t nightjar_gemm_plan_workspace_bytes(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t epilogue,
                                          int32_t kernel, int32_t split_k);
int nightjar_gemm_with_plan(int32_t dtype, const void* x, const void* w, void* y, int32_t M, int32_t N, int32_t K,
                            int32_t epilogue, int32_t kernel, int32_t split_k, void* workspace,
                            size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* NIGHTJAR_H */
