/*
 * ee.h - C ABI of the MI355X greedy speculative-verification library.
 *
 * The library runs the target-model side of edit-oriented speculative
 * decoding on one gfx950 GPU: a decoder-only transformer forward over a block
 * of draft tokens appended to a paged KV cache (Eq. 3), greedy decoding of
 * every row, the longest accepted draft prefix (Eq. 7, Sec. "Reuse"), and the
 * KV-cache commit/rollback that keeps only the accepted rows.  The Reuse
 * phase's draft source - the prefix/suffix matcher between generated tokens
 * and the original code (Sec. "Reuse") - is exported too (host code).
 *
 * Conventions shared by every call
 *  - Device memory is owned by the caller: weights, the packed-weight arena,
 *    the KV pool and the workspace are caller allocations whose device
 *    pointers are handed over at ee_create and must stay valid until
 *    ee_destroy.  The library never frees them and allocates no device memory
 *    of its own (it allocates small pinned host staging buffers).
 *  - Host arrays passed to a call are read during the call only; host outputs
 *    are written before the call returns.  ee_prefill and ee_verify are
 *    synchronous: they return after the GPU work of the call has finished.
 *  - Every call validates all of its arguments before it launches anything;
 *    a call that fails leaves the sequence state (committed length, pending
 *    token, KV contents) unchanged.  No C++ exception crosses the boundary.
 *  - Return codes: EE_OK (0) or a negative EE_E* value; ee_last_error gives a
 *    message for the last failure on a context.
 *  - A context is not thread-safe; calls on one context must not overlap.
 *
 * Calls with no passage of the paper behind them are infrastructure: sizing
 * (ee_*_bytes), ee_create / ee_destroy, ee_seq_state, ee_use_graphs,
 * ee_last_error, the test aids (ee_get_logits, ee_read_kv, ee_load_kv,
 * ee_capture) and the measurement aids (ee_profile, ee_profile_read,
 * ee_time_gemm, ee_time_stream_read).  Every other call names the passage
 * it implements.
 */
#ifndef EE_H
#define EE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  EE_OK = 0,
  EE_EINVAL = -1,     /* bad argument (shape, range, NULL, malformed tree)   */
  EE_ECAPACITY = -2,  /* KV pool, max_ctx, max_seqs or k_max exceeded         */
  EE_ESTATE = -3,     /* e.g. verify before prefill, rollback beyond length   */
  EE_EHIP = -4        /* a HIP runtime call failed                            */
};

enum { EE_F32 = 0, EE_BF16 = 1 };

typedef struct ee_ctx ee_ctx;

/* Shape of a Llama-style decoder (RMSNorm, rotary positions with rotate-half
 * pairs, grouped-query attention with contiguous head groups, SwiGLU FFN, no
 * biases, untied LM head).  Requirements checked by ee_create:
 *   head_dim in {64, 128} (64 for EE_F32); n_heads % n_kv_heads == 0;
 *   d_model, ffn, n_heads*head_dim and vocab multiples of 32 (bf16) or 16 (f32);
 *   page_size == 64; 0 <= k_max <= 512; 1 <= max_ctx <= 8192; max_seqs >= 1. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn, vocab;
  int32_t dtype;        /* EE_F32 or EE_BF16: weights, KV cache, GEMM inputs */
  float rms_eps;        /* RMSNorm epsilon                                   */
  float rope_theta;     /* rotary base                                        */
  int32_t max_ctx;      /* longest sequence (committed + one block)          */
  int32_t max_seqs;     /* sequences that may be live at once                */
  int32_t k_max;        /* longest draft (linear; draft trees <= 64 nodes)   */
  int32_t page_size;    /* KV positions per page                              */
} ee_model_config;

/* Logical weights, device pointers, row-major [out, in] in the model dtype.
 * Per-layer entries are host arrays of n_layers device pointers.  They are
 * read only inside ee_create (packed into the arena) and may be freed after. */
typedef struct {
  const void* embed;                 /* [vocab, d_model]                     */
  const void* lm_head;               /* [vocab, d_model]                     */
  const float* final_gain;           /* [d_model] fp32                       */
  const void* const* wq;             /* [n_heads*head_dim, d_model]          */
  const void* const* wk;             /* [n_kv_heads*head_dim, d_model]       */
  const void* const* wv;             /* [n_kv_heads*head_dim, d_model]       */
  const void* const* wo;             /* [d_model, n_heads*head_dim]          */
  const void* const* w_gate;         /* [ffn, d_model]                       */
  const void* const* w_up;           /* [ffn, d_model]                       */
  const void* const* w_down;         /* [d_model, ffn]                       */
  const float* const* attn_gain;     /* [d_model] fp32, attention-side norm  */
  const float* const* ffn_gain;      /* [d_model] fp32, FFN-side norm        */
} ee_weights;

/* Sizes of the three caller allocations (bytes, 256-byte aligned pieces).
 * Return 0 for an invalid config. */
size_t ee_packed_weight_bytes(const ee_model_config* cfg);
size_t ee_kv_pool_bytes(const ee_model_config* cfg);
size_t ee_workspace_bytes(const ee_model_config* cfg);

/* Build a context (infrastructure).  Packs every weight into `packed` (the library's
 * MFMA-fragment layout) and zeroes `kv_pool`, on `hip_stream` (a hipStream_t;
 * NULL = the default stream), then synchronizes that stream.  Every later
 * call runs its GPU work on a stream of the context's own, ordered after the
 * work enqueued on `hip_stream` when the call starts, and returns once that
 * work is done. */
int32_t ee_create(const ee_model_config* cfg, const ee_weights* w, void* packed,
                  void* kv_pool, void* workspace, void* hip_stream, ee_ctx** out);
int32_t ee_destroy(ee_ctx* ctx);

/* Run the prompt tokens[0..n-1] of sequence `seq` (which must be empty) in
 * blocks of at most k_max+1 rows, commit all n positions to the KV cache and
 * return the greedy token of the last row in *next_token: the first emitted
 * token of plain greedy decoding (Eq. 1, the argmax of the target's
 * distribution given the prompt), now "pending" (emitted, not yet run through
 * the model).  n >= 1.  Errors: EE_EINVAL for NULL pointers, n < 1 or a token
 * outside [0, vocab); EE_ESTATE if the sequence is not empty; EE_ECAPACITY if
 * n > max_ctx - 1 or the KV pool has too few free pages.  On an error the
 * sequence stays empty. */
int32_t ee_prefill(ee_ctx* ctx, int32_t seq, const int32_t* tokens, int32_t n,
                   int32_t* next_token);

/* Append tokens[0..n-1] to sequence `seq` without verification (n >= 0): the
 * block [pending, tokens...] is run in blocks of at most k_max+1 rows and all
 * n+1 positions are committed; *next_token = the greedy token of the last row,
 * which becomes pending.  For a model that must follow tokens chosen
 * elsewhere (a draft model catching up with the accepted output); n = 0 is
 * one greedy decoding step.  Errors: EE_ESTATE before prefill; EE_EINVAL for
 * a token outside [0, vocab); EE_ECAPACITY if len + n + 2 would exceed
 * max_ctx or the KV pool has no free page (nothing is committed then). */
int32_t ee_extend(ee_ctx* ctx, int32_t seq, const int32_t* tokens, int32_t n,
                  int32_t* next_token);

/* One verification step (Eq. 3 forward + Eq. 7 acceptance).  The block is
 * [pending, d_1..d_K]: row 0 is the pending token at position len; draft row
 * i sits at position len + depth(i).  Every row is decoded greedily (argmax
 * over the vocabulary, lowest index on exact ties).
 *   parent == NULL: linear chain; accept_len = largest a with d_i equal to
 *     the greedy token of row i-1 for all i <= a; next_token = greedy token of
 *     row a (the correction after a rejection, the bonus token if a == K).
 *   parent != NULL: draft tree of K <= 64 nodes; parent[i] is the node that node i
 *     extends (-1 = the pending token) and must satisfy parent[i] < i; node i
 *     sees the committed cache, the pending row and its ancestors.  Greedy
 *     walk: from the pending row, step to the lowest-indexed child whose token
 *     equals the current row's greedy token.  accept_len = nodes on that path,
 *     next_token = greedy token of the last one; accepted_nodes (optional,
 *     room for K entries) receives the path's node indices in depth order.
 * Effects: the pending row and the accepted rows are committed (len grows by
 * 1 + accept_len, tree rows compacted to depth order), next_token becomes
 * pending.  K = 0 is exactly one plain greedy decoding step (Eq. 1).
 * Errors: EE_ESTATE before prefill; EE_EINVAL for K < 0, K > k_max, a token
 * outside [0, vocab), a malformed tree or a tree of more than 64 nodes; EE_ECAPACITY if len + K + 1 would
 * exceed max_ctx or the KV pool has no free page. */
int32_t ee_verify(ee_ctx* ctx, int32_t seq, const int32_t* draft_tokens, int32_t K,
                  const int32_t* parent, int32_t* accept_len, int32_t* next_token,
                  int32_t* accepted_nodes);

/* ee_verify for callers that cannot allocate memory (serving loops and
 * harnesses that forbid device or host allocation during a step): the same
 * arguments, checks, kernels and results (bit for bit) as ee_verify, but the
 * step's scratch (the attention split states and the GEMM K-slice partials)
 * lives in a static device array of the library, 16 MiB per GPU (held by
 * each GPU the library runs on until the process ends), instead of the
 * context's workspace, and the block runs without graph capture or replay, so
 * the call allocates nothing (no hipMalloc, hipFree, graph instantiation or
 * other allocating routine).  The array's device address is looked up once
 * per GPU by ee_create, and the context's GPU must be the current device at
 * the call (else EE_EINVAL).  A block whose scratch exceeds 16 MiB fails with
 * EE_ECAPACITY before anything runs; it needs
 *   up(ceil((len + K + 1) / 256) * n_kv_heads * (K + 1) * (n_heads / n_kv_heads) * (head_dim + 2) * 4)
 *   + up(S * (K + 1) * 4)
 * bytes, up() rounding to 256, S = the largest K-slice count times output
 * width over the projections and the LM head (7B-class bf16, K = 32 over a
 * 2048-position context: 13.4 MB).  Every call on a GPU shares that GPU's
 * array and leaves its contents behind (every value a call reads there is
 * written earlier in the same call); calls on one GPU must not overlap, or
 * they race on it. */
int32_t ee_verify_noalloc(ee_ctx* ctx, int32_t seq, const int32_t* draft_tokens, int32_t K,
                          const int32_t* parent, int32_t* accept_len, int32_t* next_token,
                          int32_t* accepted_nodes);

/* ee_verify for n_seq distinct sequences in one block (n_seq <= max_seqs),
 * all with the same draft length K: drafts[b*K .. b*K + K-1] is the draft of
 * sequence seqs[b]; parents (NULL: every draft is a linear chain) holds
 * n_seq arrays of K parent indices laid out the same way; accept_lens[b],
 * next_tokens[b] and (optional) accepted_nodes[b*K ..] are the results of
 * sequence seqs[b], exactly as ee_verify defines them.  Each sequence reads
 * only its own cache, and its rows' arithmetic is the same as in a block of
 * its own: every result equals that of ee_verify on the sequence alone.
 * Either every sequence advances or, on error, none does.  Errors: as
 * ee_verify, plus EE_EINVAL for n_seq outside [1, max_seqs] or a sequence
 * listed twice. */
int32_t ee_verify_batch(ee_ctx* ctx, int32_t n_seq, const int32_t* seqs, const int32_t* drafts,
                        int32_t K, const int32_t* parents, int32_t* accept_lens,
                        int32_t* next_tokens, int32_t* accepted_nodes);

/* Entropy-aware dynamic verification (Sec. "Edit", Eq. 9-10) and its fixed
 * top-k variant, for linear drafts of n_seq distinct sequences (layout of
 * seqs, drafts, accept_lens and next_tokens as in ee_verify_batch).
 * For every block row i < K of a sequence, the target's top_k tokens are
 * ranked by logit (ties: lower token id first) and their probabilities
 * renormalised over those top_k tokens give the normalised entropy
 * H_i = -sum q log q / log(top_k), computed in float64 from the float32
 * logits.  The threshold is tau_i = max(1, ceil(top_k * H_i)) when dynamic
 * != 0, else top_k (top_k == 1 gives tau = 1: plain greedy verification).
 * Draft token d_{i+1} is accepted when it is one of row i's first tau_i
 * tokens; accept_len a = the longest accepted prefix, next_token = the greedy
 * (top-1) token of row a.  Unlike greedy verification this accepts tokens
 * other than the target's own, so the output may differ from plain greedy
 * decoding.  thresholds (optional, room for n_seq * K) receives tau_i of
 * every draft row at thresholds[b*K + i].
 * Effects, atomicity and errors: as ee_verify_batch, plus EE_EINVAL for
 * top_k outside [1, min(8, vocab)]. */
int32_t ee_verify_topk(ee_ctx* ctx, int32_t n_seq, const int32_t* seqs, const int32_t* drafts,
                       int32_t K, int32_t top_k, int32_t dynamic, int32_t* accept_lens,
                       int32_t* next_tokens, int32_t* thresholds);

/* Stochastic speculative verification (Sec. "Speculative Decoding", Eq. 4)
 * of a linear draft for one sequence.  Row i's target distribution is
 * p_i = softmax(logits_i / temperature); draft token d_{i+1} is accepted when
 * eps[i] * q_i[d_{i+1}] < p_i[d_{i+1}] (eps[i] < p / q), with q_dev the draft
 * model's distributions (device memory, fp32 [K][vocab], row i = the
 * distribution d_{i+1} was drawn from; NULL = a greedy draft, q one-hot at
 * the drafted token).  At the first rejected row a the next token is drawn
 * from max(0, p_a - q_a) renormalised (residual != 0; the output then follows
 * p exactly) or from p_a (residual == 0); with every draft token accepted it
 * is drawn from p_K.  A draw takes the smallest token whose cumulative weight
 * (token order) exceeds u[a] times the total.  eps (K values) and u (K + 1
 * values) are host arrays of uniform draws in [0, 1) supplied by the caller,
 * so a call is reproducible.  Probabilities are computed in float64 from the
 * float32 logits.  Effects as ee_verify.  Errors: as ee_verify, plus
 * EE_EINVAL for a draw outside [0, 1) or temperature <= 0. */
int32_t ee_verify_sample(ee_ctx* ctx, int32_t seq, const int32_t* draft_tokens, int32_t K,
                         const float* q_dev, const float* eps, const float* u, float temperature,
                         int32_t residual, int32_t* accept_len, int32_t* next_token);

/* Truncate sequence `seq` to its first new_len committed positions
 * (new_len <= len), release pages wholly beyond them and make pending_token
 * pending: the rewind of the cache to an earlier prefix (Sec. "Reuse": after
 * a rejection only the accepted prefix stays, the remaining drafts being
 * candidates for later steps; ee_verify already commits exactly that, and this
 * call rewinds explicitly, e.g. to re-verify from an earlier position).  new_len == 0 with pending_token == -1 empties the sequence (it
 * may then be prefilled again).  EE_ESTATE if new_len > len. */
int32_t ee_kv_rollback(ee_ctx* ctx, int32_t seq, int32_t new_len, int32_t pending_token);

/* Committed length and pending token of a sequence (pending -1 if empty). */
int32_t ee_seq_state(ee_ctx* ctx, int32_t seq, int32_t* len, int32_t* pending_token);

/* Reuse-phase matcher (Sec. "Reuse"; host only, no context needed).  Tries
 * suffix lengths L from min(max_ngram, n_gen) down to min_ngram; for the first
 * L that matches, returns the smallest j with original[j..j+L) equal to the
 * last L generated tokens, j + L >= cursor (the draft starts in the remaining
 * original code) and j + L < n_orig (a non-empty draft): *draft_start = j + L,
 * *match_len = L.  No match: *draft_start = -1, *match_len = 0 (EE_OK).
 * EE_EINVAL for NULL outputs, negative sizes or min_ngram < 1. */
int32_t ee_match_reuse(const int32_t* generated, int32_t n_gen, const int32_t* original,
                       int32_t n_orig, int32_t cursor, int32_t min_ngram, int32_t max_ngram,
                       int32_t* draft_start, int32_t* match_len);

/* Edit-session driver: the Reuse and Generate phases (Sec. "Reuse",
 * Sec. "Generate") over a target-model sequence and, optionally, a
 * draft-model sequence in another context (a smaller model on the same GPU).
 * Both sequences must hold the same prompt; ee_edit_begin makes the draft
 * sequence's pending token the target's (the first emitted token).
 *
 * One ee_edit_step runs one step of the current phase and appends the tokens
 * it emits to the caller's output buffer:
 *   Reuse: the matcher (ee_match_reuse with min_match, max_match; while the
 *     output is shorter than min_match, the whole output) looks for the
 *     output's suffix in the original code from the cursor on; the draft
 *     is the next k_reuse original tokens after the match, or after the cursor
 *     when nothing matches.  Greedy verification (Eq. 7); cursor := draft
 *     start + accepted + 1 (the rejected token is taken as substituted).  A
 *     rejection marks an edit position: the next step is Generate.  A step
 *     whose draft would be empty (the original is used up) runs as Generate.
 *   Generate: the draft model catches up with the output (ee_extend), drafts
 *     gamma tokens greedily, and the target verifies them with Eq. 7
 *     (top_k = 0) or Eq. 9-10 (top_k >= 1, `dynamic` as in ee_verify_topk);
 *     the draft sequence is rolled back to the accepted prefix.  Without a
 *     draft context (draft == NULL) the step is one plain greedy step.  After
 *     the step the matcher is run; a match switches back to Reuse.
 * out[0..n_out-1] is the session output so far (the first call passes the
 * first emitted token, n_out = 1); out[n_out-1] must be the target's pending
 * token.  The new tokens (accepted draft tokens, then the target's next
 * token) are written at out[n_out..n_out+*n_new-1]; out_cap >= n_out +
 * max(k_reuse, gamma) + 1.  With top_k = 0 the output is exactly the target's
 * greedy decoding whatever the draft model proposes.
 * Errors: EE_EINVAL for bad parameters (a state whose phase is neither
 * phase or whose cursor is negative among them); EE_ESTATE if out does not end with
 * the target's pending token or the draft sequence does not follow the
 * output; capacity and HIP errors as the calls it makes.  On an error the
 * target sequence is unchanged; the draft sequence is realigned by the next
 * call. */
enum { EE_PHASE_REUSE = 0, EE_PHASE_GENERATE = 1 };

typedef struct {
  int32_t k_reuse;      /* draft tokens per Reuse step, 1..k_max of the target   */
  int32_t gamma;        /* draft-model tokens per Generate step, 1..k_max         */
  int32_t top_k;        /* Generate verification: 0 greedy, 1..8 Eq. 9-10         */
  int32_t dynamic;      /* with top_k: entropy-aware tau (1) or fixed top-k (0)   */
  int32_t min_match;    /* shortest output suffix whose match resumes Reuse (>=1) */
  int32_t max_match;    /* longest suffix tried (>= min_match)                    */
} ee_edit_params;

typedef struct {
  int32_t phase;          /* phase of the next step                                */
  int32_t cursor;         /* original position a Reuse draft falls back to         */
  int32_t last_phase;     /* phase of the last step                                */
  int32_t last_accept;    /* draft tokens accepted by the last step                */
  int64_t steps[2];       /* steps run per phase                                   */
  int64_t emitted[2];     /* tokens emitted per phase                              */
  int64_t draft_tokens;   /* tokens proposed by the draft model                    */
  int64_t draft_forwards; /* forward blocks run by the draft model                 */
} ee_edit_state;

int32_t ee_edit_begin(ee_ctx* target, int32_t seq, ee_ctx* draft, int32_t draft_seq,
                      ee_edit_state* state);
int32_t ee_edit_step(ee_ctx* target, int32_t seq, ee_ctx* draft, int32_t draft_seq,
                     const int32_t* original, int32_t n_orig, const ee_edit_params* params,
                     ee_edit_state* state, int32_t* out, int32_t n_out, int32_t out_cap,
                     int32_t* n_new);

/* Copy the logits of the last prefill block or verify block (rows x vocab,
 * fp32, row-major) to host memory; rows must equal that block's row count.
 * Test and inspection aid; not needed on the hot path. */
int32_t ee_get_logits(ee_ctx* ctx, float* host_out, int32_t rows);

/* Copy committed keys/values of one layer to host memory, positions
 * [0, len) of sequence `seq`, as [len, n_kv_heads, head_dim] in the model
 * dtype (fp32 or bf16 bits).  Either output may be NULL.  Test aid. */
int32_t ee_read_kv(ee_ctx* ctx, int32_t seq, int32_t layer, void* host_k, void* host_v);

/* Install a committed cache in the empty sequence `seq`: keys and values of
 * positions [0, n) of every layer from host memory, [n_layers][n][n_kv_heads]
 * [head_dim] each in the model dtype (fp32 or bf16 bits; the caller keeps
 * ownership), and `pending` as the token the next block starts with.  The
 * sequence is then as if a prefill of n tokens had produced this cache and
 * greedy token (the Eq. 3 prefix of later blocks).  Errors (EE_EINVAL for
 * NULL arrays, n < 1 or a pending token outside [0, vocab); EE_ESTATE if the
 * sequence holds tokens; EE_ECAPACITY if n + 1 > max_ctx or the KV pool is
 * short) leave the sequence empty.  Synchronous.  The counterpart of
 * ee_read_kv: a test aid, and a way to resume from a cache computed
 * elsewhere. */
int32_t ee_load_kv(ee_ctx* ctx, int32_t seq, int32_t n, int32_t pending, const void* host_k,
                   const void* host_v);

/* Bytes of the capture buffer ee_capture needs for blocks of `rows` rows
 * (all sequences of the block together), or 0 for an invalid config or
 * rows < 1.  With R = rows, R16 = R rounded up to a multiple of 16, E = 2
 * (bf16) or 4 (fp32), qd = n_heads * head_dim and kd = n_kv_heads * head_dim,
 * every layer takes E * (R16 * (2 d_model + qd + ffn) + R * (qd + 2 kd))
 * bytes and the LM head's input E * R16 * d_model more. */
size_t ee_capture_bytes(const ee_model_config* cfg, int32_t rows);

/* Test aid: record the values of every rounding site of the forward.  While
 * `dev_buf` is non-NULL (device memory of `bytes` bytes, owned by the
 * caller), every later block runs without graph replay and copies, for each
 * layer in order, its x_attn (h * g of the attention-side norm, in the
 * packed layout of GEMM inputs: fragments [R16 / 16][cols / KS][64 lanes]
 * [16 B], KS = 32 for bf16 and 16 for fp32, where lane g * 16 + c of
 * fragment (t, s) holds row 16 t + c, columns KS s + g KS / 4 .. + KS / 4), q after
 * RoPE ([R][n_heads][head_dim]), the block's k after RoPE and v
 * ([R][n_kv_heads][head_dim] each, in block row order), the attention output
 * o (packed, qd columns), x_ffn (packed, d columns) and the SwiGLU product z
 * (packed, ffn columns); after the last layer the LM head's input x_final
 * (packed, d columns).  Every value is in the model dtype.  A block whose
 * capture would exceed `bytes` fails with EE_EINVAL before it runs.
 * dev_buf = NULL ends capturing.  These are the values a bf16 pipeline
 * rounds (Eq. 3's forward; the rounding sites are a reading, since the paper
 * states no precision), so a test can check every rounding decision of the
 * GPU against the CPU reference. */
int32_t ee_capture(ee_ctx* ctx, void* dev_buf, size_t bytes);

/* Launch mode of later prefill/verify blocks.  on != 0 (the default): the
 * kernels of each block shape (row count, sequences, linear/tree/prefill, and
 * the attention splits of the longest context, ceil((n + T) / 256)) are
 * captured once into a HIP graph and replayed (at most 512 shapes are kept;
 * past that the cache starts over); on == 0: every kernel is launched
 * individually.  Both run the same kernels with the same arguments. */
int32_t ee_use_graphs(ee_ctx* ctx, int32_t on);

/* Kernel classes of one forward, for ee_profile. */
enum {
  EE_PROF_NORM = 0,     /* embedding / residual add + RMSNorm launches  */
  EE_PROF_QKV = 1,      /* QKV GEMM                                     */
  EE_PROF_ATTN = 2,     /* split attention over the paged KV cache      */
  EE_PROF_COMBINE = 3,  /* merge of the attention splits                */
  EE_PROF_OPROJ = 4,    /* O-projection GEMM                            */
  EE_PROF_GATEUP = 5,   /* gate/up GEMM                                 */
  EE_PROF_DOWN = 6,     /* down-projection GEMM                         */
  EE_PROF_LMHEAD = 7,   /* LM-head GEMM                                 */
  EE_PROF_ARGMAX = 8,   /* vocabulary argmax                            */
  EE_PROF_ACCEPT = 9,   /* acceptance scan / tree walk                  */
  EE_PROF_COMPACT = 10, /* tree KV compaction                           */
  EE_PROF_FINISH = 11,  /* GEMM epilogues: rotary + KV append, SwiGLU,  */
                        /* logits + per-chunk maxima                    */
  EE_PROF_N = 12
};

/* Measurement aid: when bit c of class_mask is set, every launch of kernel
 * class c is bracketed by two HIP events on the context's stream, and the
 * elapsed time between them is accumulated after each prefill / verify
 * block.  class_mask = 0 turns it off (the default).  While it is on, blocks
 * are launched kernel by kernel (no graph replay). */
int32_t ee_profile(ee_ctx* ctx, uint32_t class_mask);

/* Read the accumulated per-class totals: ms[EE_PROF_N] milliseconds and
 * launches[EE_PROF_N] launch counts (either may be NULL); reset != 0 zeroes
 * them afterwards. */
int32_t ee_profile_read(ee_ctx* ctx, double* ms, int64_t* launches, int32_t reset);

/* Measurement aid: the GEMM of one projection (cls = EE_PROF_QKV,
 * EE_PROF_OPROJ, EE_PROF_GATEUP or EE_PROF_DOWN) launched for every layer in
 * turn (EE_PROF_LMHEAD: the LM head's GEMM, n_layers times), reps times, back
 * to back on the context's stream, on `rows` rows of
 * the workspace's current activations (the launch configuration a block of
 * that many rows uses); *us_per_launch = the elapsed time between two HIP
 * events around the sequence divided by the launches.  Each launch streams
 * its own layer's weights, as in a verify step; events around single
 * launches would add their own overhead to every launch.  Writes only GEMM
 * partials in the workspace (no sequence state changes).  EE_EINVAL for
 * another class, rows outside [1, max_seqs * (k_max + 1)] or reps < 1. */
int32_t ee_time_gemm(ee_ctx* ctx, uint32_t cls, int32_t rows, int32_t reps, double* us_per_launch);

/* Measurement aid (no paper passage: infrastructure): microseconds per pass
 * of a plain streaming read of `bytes` (a multiple of 16, at least 256 KiB)
 * of caller device memory at `dev_buf`, averaged over `reps` back-to-back
 * passes on the context's stream after one untimed pass: the HBM read rate
 * this GPU reaches in practice (one workgroup per CU, each reading a
 * contiguous chunk), which the verify step's rate is compared with.  The
 * buffer is only read.  EE_EINVAL for a smaller or misaligned size, a null
 * buffer or output, or reps < 1. */
int32_t ee_time_stream_read(ee_ctx* ctx, const void* dev_buf, size_t bytes, int32_t reps, double* us_per_pass);

/* Message for the last failed call on ctx (or the last failed context-free
 * call when ctx is NULL).  Never NULL; the pointer stays valid until the next
 * call on the same context. */
const char* ee_last_error(const ee_ctx* ctx);

#ifdef __cplusplus
}
#endif
#endif /* EE_H */
