/*
 * rv.h -- C ABI of the MI355X (gfx950) Reflective Verification verify pass.
 *
 * Method: "Think Before You Accept: Semantic Reflective Verification for
 * Faster Speculative Decoding" (arXiv 2505.18629).  One verify call scores,
 * in a single causal forward pass of the target model, the block
 *
 *     [c, x_1..x_k, R, ids[L-P..L-1], x_1..x_k]                (Eq. 1)
 *
 * against the cached prefix, where c = ids[L-1] is the last committed token
 * (its KV is not cached yet), x are the k draft tokens, R the reflective
 * probe ids and ids[L-P..L-1] the prefix-position tokens (Section 3.1,
 * Algorithm 1).  Block row i-1 gives the original logits o_i and block row
 * shift+i-1 the reflective logits r_i (i = 1..k+1, shift = k + |R| + P).
 * They are fused as z_i = (1 - alpha) o_i + alpha r_i (Eq. 2, Section 3.2),
 * and the exact-match rule of Algorithm 2 (Appendix A) at temperature 0
 * gives the accepted length n and the next token t = argmax z_{n+1}.
 *
 * Conventions
 *  - Every device pointer is caller-owned device memory (e.g. a torch
 *    tensor).  The library never allocates or frees device memory except
 *    the small per-cache partial-sum region it carves out of the cache
 *    buffer the caller provides.
 *  - `stream` is a hipStream_t passed as void* (NULL = default stream).
 *    Calls that take a stream are asynchronous on it; the library never
 *    synchronises the device.
 *  - Host pointers are prefixed h_, device pointers d_.
 *  - Every function validates its arguments on the host first.  On any
 *    validation failure it returns a negative rv_status and enqueues no
 *    device work; rv_last_error() then describes the failure (thread-local).
 *  - int32 token ids; ids outside [0, vocab) are detected on the device and
 *    reported per sequence (accept_len = next_id = -1).
 */
#ifndef RV_H
#define RV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RV_OK = 0,
  RV_E_ARG = -1,      /* null pointer, bad enum, size or value out of its domain */
  RV_E_RANGE = -2,    /* a prefix length outside [max(1, P), max_len] */
  RV_E_CAPACITY = -3, /* block does not fit: L - 1 + S > max_len, or S > max_block */
  RV_E_BUFFER = -4,   /* caller buffer smaller than the required byte count */
  RV_E_HIP = -5,      /* a HIP runtime call or kernel launch failed */
  RV_E_STATE = -6     /* handle used in a state that does not allow the call */
} rv_status;

enum { RV_F32 = 0, RV_BF16 = 1 };
enum { RV_RULE_GREEDY = 0, RV_RULE_TYPICAL = 1, RV_RULE_SAMPLING = 2 };
enum { RV_ENTROPY_FUSED = 0, RV_ENTROPY_ORIGINAL = 1 };
enum { RV_MAX_BATCH = 256, RV_MAX_DRAFTS = 32 };

/* Decoder shape.  Llama-style: pre-norm RMSNorm, rotate-half rotary, GQA
 * (query head h uses kv head h / (n_heads / n_kv_heads)), SwiGLU FFN,
 * untied LM head, no biases.  dtype is the storage type of the weights;
 * accumulation is fp32.  With bf16 weights every computed value that is
 * stored for a later matmul (norm outputs, queries, the KV cache, attention
 * and SwiGLU outputs) is kept as the pair hi = bf16(x), lo = bf16(x - hi) of
 * its fp32 value (about 16 significant bits), so that only the weights are
 * rounded to bf16.
 * Requirements: d_model, ffn_dim and n_heads*head_dim multiples of 128;
 * head_dim 32, 64 or 128; n_heads % n_kv_heads == 0; vocab % 16 == 0 and
 * <= 262144. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  int32_t dtype;   /* RV_F32 or RV_BF16 */
  float rms_eps;   /* RMSNorm epsilon, e.g. 1e-5 */
  float rope_base; /* rotary base, e.g. 10000 */
  float init_std;  /* std of the random-init weights, e.g. 0.02 */
} rv_config;

/* Fusion and verification parameters (Eq. 2, Table 5, Algorithms 2 and 3).
 * RV_RULE_GREEDY (Algorithm 2 at temperature 0): draft i is accepted while
 *   it equals argmax z_i.
 * RV_RULE_TYPICAL (Algorithm 3): draft i is accepted while
 *   p_i(x_i) > min(epsilon, delta * exp(-H_i)), p_i = softmax(z_i), H_i the
 *   entropy (nats) of p_i (RV_ENTROPY_FUSED) or of softmax(o_i)
 *   (RV_ENTROPY_ORIGINAL); compared in the log domain, so epsilon = +inf and
 *   delta = 0 are exact.
 * Both: n = leading accepted drafts, t = argmax z_{n+1} (lowest id on ties).
 * RV_RULE_SAMPLING (Algorithm 1, rv_verify_sampled only): see there.
 * z_i is the fused logit row divided by `temperature` (Table 5); greedy
 * decisions do not depend on it. */
typedef struct {
  float alpha;         /* weight of the reflective logits, 0 <= alpha <= 1 (Eq. 2) */
  int32_t prefix_pos;  /* P: committed tokens re-presented after the probe (Eq. 1) */
  int32_t rule;        /* RV_RULE_GREEDY, RV_RULE_TYPICAL or RV_RULE_SAMPLING */
  float epsilon;       /* typical: threshold cap, > 0 (may be +inf) */
  float delta;         /* typical: entropy-scaled threshold factor, >= 0 */
  int32_t entropy_src; /* typical: RV_ENTROPY_FUSED or RV_ENTROPY_ORIGINAL */
  float temperature;   /* > 0, finite; 1 leaves the fused logits unchanged */
} rv_fusion;

typedef struct rv_model rv_model;
typedef struct rv_cache rv_cache;

/* Status text and the calling thread's last error message. */
const char* rv_status_str(rv_status s);
const char* rv_last_error(void);

/* Bytes of device memory a model of this shape needs (weights in the packed
 * layout the kernels read, norm gains). */
rv_status rv_model_bytes(const rv_config* cfg, size_t* bytes);

/* Creates a model in the caller's buffer d_buf (>= rv_model_bytes) and fills
 * it with seeded random-init weights (the paper's trained targets are not
 * available).  Element (r, c) of logical matrix t (0 embedding,
 * 1+7l+{q,k,v,o,gate,up,down}, 1+7L LM head) has index i = r*in + c and value
 *   h = mix(((t << 36) + i) ^ mix(seed)),  mix(x) = splitmix64 finaliser of
 *       x + 0x9E3779B97F4A7C15 (Steele, Lea, Flood, OOPSLA 2014);
 *   s = sum of the four 16-bit fields of h - 2*65535;
 *   w = fp32(s) * fp32(init_std / sqrt(4 (65536^2 - 1) / 12)), then RNE to dtype.
 * Norm gains are 1.  Asynchronous on stream.  *out is a host handle; free it
 * with rv_model_free (which does not touch d_buf). */
rv_status rv_init_weights(const rv_config* cfg, uint64_t seed, void* d_buf, size_t buf_bytes,
                          void* stream, rv_model** out);
void rv_model_free(rv_model* m);

/* Bytes of device memory for a cache of `batch` sequences of up to max_len
 * positions: the KV cache [layer][b][kv_head] x (max_len rounded up to a
 * multiple of 64) positions x head_dim (fp32 row-major; for bf16 models a
 * bf16 hi plane plus a bf16 lo plane, value = hi + lo, each in the order the
 * attention kernel reads it -- rv_debug_export_kv returns rows), the
 * token-id history [b][max_len] (int32), the rotary table and the per-call
 * workspace for blocks of up to max_block rows per sequence and up to
 * max_drafts draft tokens. */
rv_status rv_cache_bytes(const rv_model* m, int32_t batch, int32_t max_len, int32_t max_block,
                         int32_t max_drafts, size_t* bytes);

/* Creates a cache handle over d_buf (>= rv_cache_bytes).  Uploads the rotary
 * table (synchronously) and zeroes the buffer.  The model must outlive it. */
rv_status rv_cache_create(rv_model* m, int32_t batch, int32_t max_len, int32_t max_block,
                          int32_t max_drafts, void* d_buf, size_t buf_bytes, rv_cache** out);
void rv_cache_free(rv_cache* c);

/* Prefill.  d_prefix_ids is [batch][ld] int32 on the device; sequence b has
 * h_prefix_len[b] committed tokens (1 <= L_b <= max_len, L_b <= ld).  Stores
 * ids[0..L_b-1] in the id history and the KV of positions 0..L_b-2 (the
 * last committed token is left for the first verify, which scores it as
 * block row 0).  Asynchronous on stream. */
rv_status rv_prefill_cache(rv_cache* c, const int32_t* d_prefix_ids, int32_t ld,
                           const int32_t* h_prefix_len, void* stream);

/* One verification pass (Algorithm 1 with the rule of Algorithm 2 or 3).
 *   h_prefix_len [batch]  host: committed length L_b of each sequence;
 *                         requires max(1, P) <= L_b and L_b - 1 + S <= max_len,
 *                         S = 1 + 2k + n_probe + P <= max_block.
 *   d_draft_ids [batch][k] device int32, 0 <= k <= max_drafts.
 *   d_probe_ids [n_probe]  device int32, shared by all sequences (may be
 *                          NULL when n_probe == 0).
 *   fusion                 alpha in [0, 1], P >= 0, rule RV_RULE_GREEDY or
 *                          RV_RULE_TYPICAL (then epsilon > 0, delta >= 0, not
 *                          NaN, entropy_src RV_ENTROPY_*).
 *   d_accept_len, d_next_id [batch] device int32 outputs: n_b and t_b, or
 *                          -1 and -1 if any id the block uses is out of range.
 * Side effects: writes KV at positions L_b-1 .. L_b-2+S (only L_b-1 ..
 * L_b-1+n_b remain meaningful, the rest is overwritten by later calls, which
 * prunes the template and second-copy entries, Section 3.1) and appends
 * x_1..x_n, t to the id history at L_b .. L_b+n.  The caller's next prefix
 * length is L_b + n_b + 1.  Repeating a call with the same arguments gives
 * the same outputs.  Asynchronous on stream. */
rv_status rv_verify(rv_cache* c, const int32_t* h_prefix_len, const int32_t* d_draft_ids, int32_t k,
                    const int32_t* d_probe_ids, int32_t n_probe, const rv_fusion* fusion,
                    int32_t* d_accept_len, int32_t* d_next_id, void* stream);

/* rv_verify with a draft count per sequence (dynamic draft length).
 *   d_draft_ids [batch][ld_drafts] device int32; sequence b uses its first
 *               h_draft_len[b] entries (0 <= h_draft_len[b] <= ld_drafts <=
 *               max_drafts).
 *   h_draft_len [batch] host int32.
 * Sequence b's block has S_b = 1 + 2 k_b + n_probe + P rows; the probe, P,
 * alpha and the rule (RV_RULE_GREEDY or RV_RULE_TYPICAL) are shared.
 * Per-row debug outputs then hold sum_b (k_b + 1) rows, sequence after
 * sequence.  Everything else as rv_verify. */
rv_status rv_verify_ragged(rv_cache* c, const int32_t* h_prefix_len, const int32_t* d_draft_ids, int32_t ld_drafts,
                           const int32_t* h_draft_len, const int32_t* d_probe_ids, int32_t n_probe,
                           const rv_fusion* fusion, int32_t* d_accept_len, int32_t* d_next_id, void* stream);

/* Overwrites the id history: ids[b][h_pos[b]] = d_ids[b] for every sequence
 * b with h_pos[b] >= 0 (host int32 [batch]; device int32 [batch]).  A
 * speculative loop uses it to commit the token the target emitted into the
 * draft model's cache (whose own history holds the draft token there); the
 * next call on that cache then scores it as block row 0.  Positions must be
 * < max_len.  Asynchronous. */
rv_status rv_commit_tokens(rv_cache* c, const int32_t* h_pos, const int32_t* d_ids, void* stream);

/* rv_verify with Algorithm 1's speculative-sampling rule (fusion->rule must
 * be RV_RULE_SAMPLING).
 *   d_draft_probs [batch][k][vocab] device fp32: the draft distributions q_i
 *                 the drafts were sampled from (rows sum to 1; not checked).
 *                 May be NULL when k == 0.
 *   seed          key of the random numbers; a call is a pure function of
 *                 its inputs and seed, so callers vary the seed per step.
 * With p_i = softmax(z_i): draft i is rejected when r_i * q_i(x_i) >
 * p_i(x_i) (r_i uniform); n = leading accepted drafts; t is drawn from
 * norm(max(0, p_{n+1} - q_{n+1})) if n < k, else from p_{k+1}, as
 * argmax_v (log w_v - log(-log u_v)) (Gumbel-max).  Random numbers:
 * Philox4x64-10 (Salmon et al., SC 2011) with key (seed, 0); r_i is word 0
 * at counter (i, b, 0, 0) and u_v word v % 4 at counter (v / 4, b, 1, 0),
 * b the batch slot; a 64-bit word w becomes ((w >> 41) + 1/2) / 2^23.
 * Everything else as rv_verify. */
rv_status rv_verify_sampled(rv_cache* c, const int32_t* h_prefix_len, const int32_t* d_draft_ids, int32_t k,
                            const float* d_draft_probs, const int32_t* d_probe_ids, int32_t n_probe,
                            const rv_fusion* fusion, uint64_t seed, int32_t* d_accept_len,
                            int32_t* d_next_id, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * decision of rv_debug_fuse_accept -- accept_len and next_id, the same
 * kernels and bits -- without a cache.  No id history is written and no
 * per-row outputs are kept.  Its scratch (per-chunk softmax statistics,
 * merged row statistics, margins) is a static device array of
 * RV_NOALLOC_SCRATCH_BYTES that each GPU the library runs on holds until the
 * process ends; the call allocates nothing.
 *   d_logits [batch][2(k+1)][vocab] device fp32, as rv_debug_fuse_accept.
 *   batch in [1, RV_MAX_BATCH], k in [0, RV_MAX_DRAFTS], vocab in [1, 262144],
 *   and batch * (k+1) * ceil(vocab / 2048) <= 65536 (else RV_E_CAPACITY).
 *   d_draft_ids [batch][k] device int32 (NULL if k == 0).
 *   fusion: rule RV_RULE_GREEDY or RV_RULE_TYPICAL.
 * Every call on one GPU uses that GPU's one array: calls that overlap on a
 * GPU (other streams, other host threads) race and must be serialised by the
 * caller.  Asynchronous on stream. */
#define RV_NOALLOC_SCRATCH_BYTES (4718592)
rv_status rv_fuse_accept_noalloc(const float* d_logits, int32_t batch, int32_t k, int32_t vocab,
                                 const int32_t* d_draft_ids, const rv_fusion* fusion, int32_t* d_accept_len,
                                 int32_t* d_next_id, void* stream);

/* ---- inspection (tests and benchmarks) ---- */

/* The fusion, log-softmax and accept stage of rv_verify (Eq. 2; Algorithm 2,
 * or Algorithm 3 with RV_RULE_TYPICAL; Appendix A) run by the same kernels
 * on logits the caller supplies instead of the LM head's.
 *   d_logits [batch][2(k+1)][vocab] device fp32: per sequence the original
 *                rows o_1..o_{k+1}, then the reflective rows r_1..r_{k+1};
 *                copied into the cache's logit rows.  Entries may be -inf
 *                (an id ruled out) as long as every row has a finite entry;
 *                where alpha is 0 or 1 the row weighted by 0 must be finite
 *                (0 * inf is NaN in Eq. 2 as written).
 *   h_prefix_len [batch] host: L_b; the decision is appended to the id
 *                history at L_b .. L_b+n as rv_verify does (1 <= L_b and
 *                L_b + k + 1 <= max_len).
 *   d_draft_ids [batch][k] device int32 (NULL if k == 0), k <= max_drafts; a
 *                sequence with an id outside [0, vocab) gets -1, -1.
 *   fusion       as rv_verify (prefix_pos is not used; the sampling rule is
 *                not available here).
 * rv_debug_output then returns the rows of this call.  Asynchronous. */
rv_status rv_debug_fuse_accept(rv_cache* c, const float* d_logits, const int32_t* h_prefix_len,
                               const int32_t* d_draft_ids, int32_t k, const rv_fusion* fusion, int32_t* d_accept_len,
                               int32_t* d_next_id, void* stream);

/* Which result of the last verify to copy.  Per-row results have one row per
 * (sequence b, i = 1..k_b+1), sequence after sequence ([batch][k+1] when every
 * sequence has k drafts).  RV_OUT_ORIG .. RV_OUT_LOGP_FUSED are fp32 rows of
 * vocab entries: raw logits o_i and r_i, fused logits z_i, and their
 * log-softmax (natural log).  RV_OUT_ENTROPY is fp32 [2][rows]: the entropy
 * (nats) of softmax(z_i), then of softmax(o_i).  RV_OUT_MARGINS is fp32
 * [batch][k+2] (k the draft-id stride): for each tested draft the distance of
 * its decision from the boundary (greedy: z_i[x_i] - max_{v != x_i} z_i[v];
 * typical: log p_i(x_i) - log threshold_i; sampling: log p_i(x_i) -
 * log(r_i q_i(x_i)); NaN for untested drafts), NaN, and last the top-1
 * minus top-2 gap of z_{n+1} (sampling: of the perturbed draw scores).
 * RV_OUT_PROB_FUSED is the fused distribution p_i = softmax(z_i) itself
 * (exp of RV_OUT_LOGP_FUSED), e.g. the draft distributions q_i a sampling
 * draft model hands to rv_verify_sampled. */
enum {
  RV_OUT_ORIG = 0, RV_OUT_REFL = 1, RV_OUT_FUSED = 2,
  RV_OUT_LOGP_ORIG = 3, RV_OUT_LOGP_REFL = 4, RV_OUT_LOGP_FUSED = 5,
  RV_OUT_ENTROPY = 6, RV_OUT_MARGINS = 7, RV_OUT_PROB_FUSED = 8
};

/* Copies one result of the last verify into d_dst (at least the byte size
 * of that result).  RV_E_STATE if no verify ran on this cache.
 * Asynchronous. */
rv_status rv_debug_output(const rv_cache* c, int32_t which, float* d_dst, size_t dst_bytes, void* stream);

/* Copies K and V of one (layer, sequence) for positions [pos0, pos0+npos)
 * into d_k and d_v.  fp32 models: [kv_head][npos][head_dim] fp32 each.
 * bf16 models: [2][kv_head][npos][head_dim] bf16 each, the hi plane then the
 * lo plane (the cached value is hi + lo).  Asynchronous. */
rv_status rv_debug_export_kv(const rv_cache* c, int32_t layer, int32_t seq, int32_t pos0, int32_t npos,
                             void* d_k, void* d_v, size_t dst_bytes, void* stream);

/* Copies ids[seq][pos0 .. pos0+n) of the id history into d_dst. Asynchronous. */
rv_status rv_debug_export_ids(const rv_cache* c, int32_t seq, int32_t pos0, int32_t n, int32_t* d_dst,
                              void* stream);

/* Stored bits of logical weight elements (synchronous; for bit-equality
 * checks of the generator).  tensor: 0 embedding, 1+7l+{q,k,v,o,gate,up,down},
 * 1+7L LM head.  h_idx are flat logical indices r*in + c.  Bits are the bf16
 * pattern in the low half, or the fp32 pattern. */
rv_status rv_debug_weight_bits(const rv_model* m, int32_t tensor, const int64_t* h_idx, int32_t n,
                               uint32_t* h_bits);

/* Intermediate activations of the last prefill or verify pass, for the
 * rows of that pass (row r = b*S + j for a verify block).  The values are
 * those of the final layer:
 *   RV_WS_RESID   fp32 [rows][d_model]     residual stream: after a prefill, after the
 *                 last layer; after a verify, before the last layer's down
 *                 projection (the final norm adds that projection's k-group
 *                 partials as it reads the rows the LM head needs)
 *   RV_WS_ATTN    operand [rows][n_heads*head_dim]  attention output (pre o-proj)
 *   RV_WS_ACT     operand [rows][ffn_dim]  SwiGLU output (pre down-proj)
 *   RV_WS_QUERY   operand [rows][n_heads*head_dim]  rotated queries
 * A matmul operand of a bf16 model is the pair hi = bf16(x), lo = bf16(x - hi)
 * of its fp32 value x; it is copied as the hi plane followed by the lo plane
 * ([2][rows][width] bf16).  fp32 models copy [rows][width] fp32.
 * Asynchronous. */
enum { RV_WS_RESID = 0, RV_WS_ATTN = 1, RV_WS_ACT = 2, RV_WS_QUERY = 3 };
rv_status rv_debug_workspace(const rv_cache* c, int32_t which, int32_t rows, void* d_dst, size_t dst_bytes,
                             void* stream);

/* Kernel classes of the event profiler. */
enum {
  RV_PROF_PLAN = 0, RV_PROF_NORM = 1, RV_PROF_QKV = 2, RV_PROF_ATTN = 3, RV_PROF_COMBINE = 4, RV_PROF_O = 5,
  RV_PROF_GATEUP = 6, RV_PROF_DOWN = 7, RV_PROF_LMHEAD = 8, RV_PROF_TAIL = 9, RV_PROF_NCLASS = 10
};

/* enable != 0: discard earlier records and, from now on, record a HIP event
 * pair on the call's stream around every kernel launch of prefill and verify
 * (the events add a little time between launches, so timing runs keep this
 * off).  enable == 0 stops recording. */
rv_status rv_debug_profile(rv_cache* c, int32_t enable);

/* Sum of the recorded durations (ms) and number of launches of one kernel
 * class.  The caller must have synchronised the stream. */
rv_status rv_debug_profile_read(const rv_cache* c, int32_t kclass, double* total_ms, int32_t* launches);

/* Fused matrices as the kernels store them. */
enum { RV_MAT_QKV = 0, RV_MAT_O = 1, RV_MAT_GATEUP = 2, RV_MAT_DOWN = 3, RV_MAT_LM_HEAD = 4 };

/* Average duration (ms) of the production kernel of one matrix class
 * (RV_MAT_O, RV_MAT_GATEUP, RV_MAT_DOWN or RV_MAT_LM_HEAD), launched `reps`
 * times back to back on `stream` with the launch shape and epilogue a verify
 * pass of M rows uses, cycling through the layers' weights (so no launch
 * re-reads cached weights), timed with HIP events around the whole batch.
 * Reads the workspace operands as they are and overwrites workspace outputs
 * (residual stream, logits, partials); the KV cache and the id history are
 * untouched.  Synchronous. */
rv_status rv_debug_time_matrix(rv_cache* c, int32_t matrix, int32_t M, int32_t reps, void* stream, float* avg_ms);

/* Y[M][N] = X[M][K] . W^T with the production matrix kernel, for one stored
 * matrix (layer is ignored for RV_MAT_LM_HEAD).  Columns of Y are in logical
 * order: QKV = [q rows; k rows; v rows], GATEUP = [gate rows; up rows].
 * X is the operand form: for bf16 models two planes [2][M][K] bf16 (hi then
 * lo; X = hi + lo), for fp32 models [M][K] fp32.  Y is fp32 [M][N].
 * M <= the cache's row capacity.  Asynchronous. */
rv_status rv_debug_linear(const rv_cache* c, int32_t layer, int32_t matrix, const void* d_x, int32_t M,
                          float* d_y, size_t y_bytes, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* RV_H */
