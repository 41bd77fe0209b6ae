// Kernel argument blocks and launchers shared by the host orchestration and
// the kernel translation units.
#pragma once
#include "rv_common.h"
#include "rv_plan.h"

// ---------------------------------------------------------------- init
hipError_t launch_init_packed(int dtype, void* dst, const MatDesc& md, uint64_t t0, uint64_t t1, uint64_t t2,
                              int r1, int r2, uint64_t seed_mix, float scale, hipStream_t st);
hipError_t launch_init_rowmajor(int dtype, void* dst, uint64_t tensor, size_t n, uint64_t seed_mix, float scale,
                                hipStream_t st);
hipError_t launch_fill_f32(float* dst, float v, size_t n, hipStream_t st);

// ---------------------------------------------------------------- profiling
// When set, the next matrix-kernel launch on this thread records these events
// at its own start and end (hipExtLaunchKernelGGL) and clears them.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
extern thread_local LaunchEvents g_launch_events;

// ---------------------------------------------------------------- matrix kernel
enum EpiKind {
  EPI_STORE = 0,          // Y[t][p] = acc                        (fp32)
  EPI_RESID = 1,          // Y[t][p] += acc                       (fp32 residual stream)
  EPI_SWIGLU = 2,         // act = operand(silu(gate) * up)       (gate/up tile pairs)
  EPI_QKV = 3,            // rotary on q/k, q -> operand, k/v -> KV cache
  EPI_STORE_LOGICAL = 4,  // Y[t][logical(p)] = acc               (inspection)
  EPI_PARTIAL = 5,        // P[kg][t][p] = partial over k-group kg (summed by the next RMSNorm)
};

struct GemmArgs {
  const void* W;      // packed matrix
  const void* X;      // operand tiles [M/16][K/KT][64][16 B]: bf16 hi plane, or fp32;
  const void* X2;     //   bf16 lo plane; token tiles up to the launch's token groups are read
  int M, N, K;
  int n_tg;           // token groups of MTT*16 tokens
  int gk;             // k-groups; (K/KT) % (4*gk) == 0
  float* Y;           // STORE / RESID / STORE_LOGICAL output, leading dim ldy
  int ldy;
  float* P;           // PARTIAL output [gk][M][ldy]
  void* act;          // SWIGLU output operand [rows][N/2] (hi plane / fp32)
  void* act2;         // lo plane
  int ld_act;
  // EPI_QKV
  void* qbuf;         // rotated q operand [rows][Hq*hd] (hi plane / fp32)
  void* qbuf2;        // lo plane
  void* kc;           // this layer's K cache [B][Hkv][kv_len x hd] (layout: put_k4): hi plane (or fp32)
  void* vc;
  void* kc2;          // lo planes (bf16 models)
  void* vc2;
  const int* row_pos;
  const int* row_seq;
  const float* rope_cos;  // [max_len][hd/2]
  const float* rope_sin;
  int hd, n_heads, n_kv, kv_len, q_rows, k_rows;
  MatDesc md;
};
// nt: row tiles per workgroup (1, 2, 4 or 8, and 3 or 6 for EPI_PARTIAL; even for SWIGLU);
// mtt: token tiles (1, 2, 4; 1 or 2 with nt = 8).
hipError_t launch_gemm(int dtype, int epi, const GemmArgs& a, int nt, int mtt, hipStream_t st);
// bf16, many tokens: nw*nt*16 rows x mt*16 tokens per workgroup of nw waves ((nw, nt, mt)
// one of (8, 4, 8), (8, 4, 4), (8, 2, 8), (8, 2, 4), (8, 2, 6), (12, 2, 4)), n_tg = ceil(M / (mt*16))
// token groups; N % (16*nw*nt) == 0; gk k-groups of a multiple of 4 k-steps each (gk > 1
// only with EPI_PARTIAL).
hipError_t launch_gemm_tiled(int epi, const GemmArgs& a, int nw, int nt, int mt, hipStream_t st);

// ---------------------------------------------------------------- attention
// Query rows of one pass are grouped in segments (one per sequence and
// chunk): rows row0 .. row0+n-1 of the row plan at positions pos0 .. pos0+n-1
// of sequence b.  Query q of (segment, kv head) is row q / G, head kv*G + q % G.
struct AttnArgs {
  const void* q;        // rotated q operand [rows][Hq*hd] (hi plane / fp32)
  const void* q2;       // lo plane
  const void* kc;       // layer base of the K cache: hi plane (or fp32); [B][Hkv][kv_len x hd], layout: put_k4
  const void* vc;
  const void* kc2;      // lo planes (bf16 models)
  const void* vc2;
  const int* seg_b;
  const int* seg_row0;
  const int* seg_n;
  const int* seg_pos0;
  int nseg;
  int n_heads, n_kv, hd, kv_len;
  int ks;               // keys per split (multiple of 64)
  int nsplit;
  int qmax;             // query stride per (segment, kv head) in the partial buffers
  float* part_o;        // [nsplit][nseg*Hkv][qmax][hd]
  float* part_ml;       // [nsplit][nseg*Hkv][qmax][2]  (running max in log2 units, sum)
  void* out;            // attention output operand [rows][Hq*hd] (hi plane / fp32)
  void* out2;           // lo plane
  float scale_log2;     // log2(e) / sqrt(hd)
};
// qpw: queries per workgroup (plan_attn_queries; 192 for bf16 only), n_qgroups = ceil(qmax / qpw).
hipError_t launch_attention(int dtype, const AttnArgs& a, int n_qgroups, int qpw, hipStream_t st);
hipError_t launch_attn_combine(int dtype, const AttnArgs& a, hipStream_t st);
// Copies positions pos0 .. pos0+npos-1 of every kv head of one sequence out of
// a bf16 K (is_v false) or V cache block into row-major planes
// dst[2][n_kv][npos][hd] (hi, lo).  src: the sequence's first (kv head) block.
hipError_t launch_export_kv(const void* src_hi, const void* src_lo, int hd, int n_kv, int kv_len, int pos0,
                            int npos, bool is_v, void* dst, hipStream_t st);

// ---------------------------------------------------------------- norms and planning
// RMSNorm of rows of the fp32 residual h into matmul operands (out, out2).  Output row r
// reads source row gather[r] (gather != NULL: the rows the LM head needs) or r.
// With P != NULL the source row first takes h += sum over g < gk of P[g][row]
// (k-group order; P holds p_rows rows per k-group): the pending partials of
// the previous matmul.  Without a gather h is written back; with one it is
// only read (output rows may share a source row).
hipError_t launch_rmsnorm(int dtype, float* h, int rows, int d, const float* gain, float eps, void* out,
                          void* out2, const int* gather, const float* P, int gk, int p_rows, hipStream_t st);

// Per-sequence draft counts k_b of a verify pass (uniform passes have k_b = k).
// Block b has S_b = 1 + 2 k_b + n_probe + P rows from row b (1 + n_probe + P)
// + 2 K_b, and k_b + 1 fused rows from row b + K_b, with K_b = sum_{b' < b} k_b'.
RV_DEV inline int kb_prefix(const uint8_t* kb, int b) {
  int s = 0;
  for (int i = 0; i < b; ++i) s += kb[i];
  return s;
}

struct QkvFinish {
  const float* P;        // [gk][M][N] partials of the packed QKV matrix (physical rows)
  int gk, M, N;
  int q_rows, k_rows, hd, n_heads, n_kv, kv_len;
  const int* row_pos;
  const int* row_seq;
  const float* rope_cos;
  const float* rope_sin;
  void* qbuf;
  void* qbuf2;
  void* kc;
  void* vc;
  void* kc2;
  void* vc2;
};
hipError_t launch_qkv_finish(int dtype, const QkvFinish& a, hipStream_t st);


// Converts operand planes between row-major [rows][K] and operand tiles.
hipError_t launch_retile(int dtype, const void* src, void* dst, int rows, int K, bool to_tiles, hipStream_t st);

struct PlanVerify {
  int B, S, k, n_probe, P, d, V, max_len;  // S: largest block, k: draft-id stride
  const int* ids;        // history [B][max_len]
  const int* drafts;     // [B][k], sequence b uses the first kb[b]
  int* lm_src;           // [sum 2(k_b+1)]: block row feeding each LM-head row
  const int* probe;      // [n_probe]
  const void* embed;     // [V][d] T
  float* h;              // [rows][d]
  int* row_pos;
  int* row_seq;
  int* row_bad;          // [rows]: 1 if the row's id is out of range
  int* seg_b;
  int* seg_row0;
  int* seg_n;
  int* seg_pos0;
  int L[RV_MAX_BATCH];
  uint8_t kb[RV_MAX_BATCH];
};
hipError_t launch_plan_verify(int dtype, const PlanVerify& p, hipStream_t st);

struct PlanPrefill {
  int nseg, rows, d, V, ld;
  const int* prefix;     // [B][ld]
  const void* embed;
  float* h;
  int* row_pos;
  int* row_seq;
  int* seg_b;
  int* seg_row0;
  int* seg_n;
  int* seg_pos0;
  int sb[RV_MAX_SEGS], spos0[RV_MAX_SEGS], sn[RV_MAX_SEGS], srow0[RV_MAX_SEGS];
};
hipError_t launch_plan_prefill(int dtype, const PlanPrefill& p, hipStream_t st);

struct StoreIds {
  int B, ld, V, max_len;
  const int* prefix;
  int* ids;
  int* seq_bad;
  int L[RV_MAX_BATCH];
};
hipError_t launch_store_ids(const StoreIds& s, hipStream_t st);

// ---------------------------------------------------------------- LM-head tail
struct HeadArgs {
  int B, k, V, max_len, nchunk, chunk;  // k: largest draft count (draft-id and margin stride k + 2)
  int n_probe, P, R1;                   // R1 = sum (k_b + 1) fused rows
  float alpha;
  int rule;              // RV_RULE_GREEDY / RV_RULE_TYPICAL
  float eps, delta;      // typical threshold parameters
  int ent_src;           // RV_ENTROPY_FUSED / RV_ENTROPY_ORIGINAL
  float temp;            // fused logits are divided by it (1: unchanged)
  const float* q;        // sampling: draft distributions [B][k][V]
  uint64_t seed;         // sampling: Philox key word 0
  const float* logits;   // per sequence 2(k_b+1) rows: o rows then r rows
  float* z;              // [R1][V], sequence b from row b + K_b; NULL: not kept (greedy/typical rules)
  float* part;           // [4][R1][nchunk][4]: (max, sum, centred sum) of o, r, z; z's top-2
  float* lse;            // [3][R1]
  float* entropy;        // [2][R1]: entropy of softmax(z), then of softmax(o)
  float* lp;             // [3][R1][V]: log-softmax of o, r, z; NULL: not written
  float* margins;        // [B][k+2]: margins of tested drafts, then top1-top2 gap last
  const int* drafts;     // [B][k]
  int* ids;              // history [B][max_len]; NULL: the decision is not appended
  const int* row_bad;    // [block rows], or NULL: logits given by the caller (draft ids checked instead)
  const int* seq_bad;    // [B] (with row_bad)
  int* accept_len;
  int* next_id;
  int* argmax;           // [R1]
  int L[RV_MAX_BATCH];
  uint8_t kb[RV_MAX_BATCH];
};
hipError_t launch_head(const HeadArgs& a, hipStream_t st);
// dst[i] = exp(src[i]) for i < n.
hipError_t launch_exp(const float* src, float* dst, size_t n, hipStream_t st);

// ---------------------------------------------------------------- host helpers
// Records the calling thread's error message (rv_last_error) and returns s.
rv_status rv_fail(rv_status s, const char* fmt, ...);
// Validation of the fusion parameters shared by the verify entry points.
rv_status rv_check_fusion(const rv_fusion* fusion);
