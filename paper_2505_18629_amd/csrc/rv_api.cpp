// Host side of the C ABI: argument validation, device-memory layout inside
// caller buffers, and the launch sequence of prefill and verify.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "rv_internal.h"

namespace {

thread_local std::string g_err;

}  // namespace

rv_status rv_fail(rv_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

namespace {


rv_status hip_fail(hipError_t e, const char* what) {
  return rv_fail(RV_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                 \
  do {                                      \
    hipError_t e_ = (expr);                 \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

constexpr size_t kAlign = 256;
constexpr int kVocabChunk = 2048;    // vocabulary chunk of the LM-head tail (8 entries per thread)

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
int round_up(int x, int a) { return (x + a - 1) / a * a; }

// Bump allocator used both to size a buffer and to carve it.
struct Carve {
  char* base;
  size_t off = 0;
  explicit Carve(void* b) : base((char*)b) {}
  template <class P> P take(size_t bytes) {
    off = align_up(off, kAlign);
    P p = (P)(base ? base + off : nullptr);
    off += bytes;
    return p;
  }
};

uint64_t splitmix_finalise(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

}  // namespace

struct rv_model {
  rv_config cfg;
  uint64_t seed;
  char* base;
  size_t bytes;
  int es;
  MatDesc qkv, o, gateup, down, lm;
  void* embed;
  float* norm_f;
  void* lm_head;
  std::vector<void*> w_qkv, w_o, w_gateup, w_down;
  std::vector<float*> n1, n2;
};

struct rv_cache {
  rv_model* m;
  int B, max_len, max_block, max_drafts;
  int kv_len;  // cached positions per (sequence, kv head): max_len rounded up to whole 64-key tiles
  char* base;
  size_t bytes;
  int rows_cap, out_rows_cap, r1_cap, nchunk;
  size_t kv_layer_elems;
  char* kc;   // K cache [layer][b][kv_head][kv_len x hd] (order: put_k4 / put_v4): bf16 hi plane, or fp32
  char* vc;
  char* kc2;  // bf16 lo planes (bf16 models)
  char* vc2;
  int* ids;
  float* rope_cos;
  float* rope_sin;
  int* seq_bad;
  int *row_pos, *row_seq, *row_bad;
  int *seg_b, *seg_row0, *seg_n, *seg_pos0;
  float* h;
  // matmul operands: first plane (bf16 hi, or fp32) and bf16 lo plane
  void *xn, *xn2, *qbuf, *qbuf2, *att, *att2, *act, *act2, *lm_x, *lm_x2;
  size_t part_entries;
  float *part_o, *part_ml;
  float* gpart;  // k-group partials of a split matmul [gk][rows][max(d_model, qkv rows)], gk*rows <= gpart_rows
  int gpart_rows;
  float *logits, *z, *lp, *hpart, *lse, *margins, *entropy;
  int* lm_src;                      // block row of each LM-head row of the last verify
  int last_R1;                      // fused rows of the last verify
  uint8_t last_kb[RV_MAX_BATCH];    // its per-sequence draft counts
  int* argmax;
  int last_k = -1;
  // event profiler
  bool prof = false;
  std::vector<hipEvent_t> prof_ev;   // pairs: start, stop
  std::vector<int> prof_cls;
  size_t prof_used = 0;
  ~rv_cache() {
    for (hipEvent_t e : prof_ev) (void)hipEventDestroy(e);
  }
};

namespace {

rv_status check_config(const rv_config* c) {
  if (!c) return rv_fail(RV_E_ARG, "config is NULL");
  if (c->dtype != RV_F32 && c->dtype != RV_BF16) return rv_fail(RV_E_ARG, "dtype must be RV_F32 or RV_BF16");
  if (c->n_layers <= 0 || c->d_model <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 || c->ffn_dim <= 0 ||
      c->vocab <= 0)
    return rv_fail(RV_E_ARG, "shape fields must be positive");
  if (c->vocab > 64 * 2 * 2048) return rv_fail(RV_E_ARG, "vocab must be <= 262144");
  if (c->d_model % 128 || c->ffn_dim % 128 || (c->n_heads * c->head_dim) % 128)
    return rv_fail(RV_E_ARG, "d_model, ffn_dim and n_heads*head_dim must be multiples of 128");
  if (c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 128)
    return rv_fail(RV_E_ARG, "head_dim must be 32, 64 or 128");
  if (c->n_heads % c->n_kv_heads) return rv_fail(RV_E_ARG, "n_heads must be a multiple of n_kv_heads");
  if (c->vocab % 16) return rv_fail(RV_E_ARG, "vocab must be a multiple of 16");
  if ((long long)c->vocab * c->d_model >= (1LL << 36)) return rv_fail(RV_E_ARG, "tensor too large for the generator");
  if (!(c->rms_eps > 0.f) || !(c->rope_base > 1.f) || !(c->init_std > 0.f))
    return rv_fail(RV_E_ARG, "rms_eps, init_std must be > 0 and rope_base > 1");
  return RV_OK;
}

void describe(rv_model* m) {
  const rv_config& c = m->cfg;
  const int qd = c.n_heads * c.head_dim, kvd = c.n_kv_heads * c.head_dim;
  m->qkv = MatDesc{MAT_QKV, qd + 2 * kvd, c.d_model, c.head_dim, qd, kvd};
  m->o = MatDesc{MAT_PLAIN, c.d_model, qd, c.head_dim, 0, 0};
  m->gateup = MatDesc{MAT_GATEUP, 2 * c.ffn_dim, c.d_model, c.head_dim, 0, 0};
  m->down = MatDesc{MAT_PLAIN, c.d_model, c.ffn_dim, c.head_dim, 0, 0};
  m->lm = MatDesc{MAT_PLAIN, c.vocab, c.d_model, c.head_dim, 0, 0};
}

size_t mat_bytes(const MatDesc& d, int es) { return (size_t)d.N * d.K * es; }

// Lays the model out in `buf` (or only sizes it when buf is NULL).
size_t model_layout(rv_model* m, void* buf) {
  const rv_config& c = m->cfg;
  Carve cv(buf);
  m->embed = cv.take<void*>((size_t)c.vocab * c.d_model * m->es);
  m->w_qkv.assign(c.n_layers, nullptr);
  m->w_o.assign(c.n_layers, nullptr);
  m->w_gateup.assign(c.n_layers, nullptr);
  m->w_down.assign(c.n_layers, nullptr);
  m->n1.assign(c.n_layers, nullptr);
  m->n2.assign(c.n_layers, nullptr);
  for (int l = 0; l < c.n_layers; ++l) {
    m->w_qkv[l] = cv.take<void*>(mat_bytes(m->qkv, m->es));
    m->w_o[l] = cv.take<void*>(mat_bytes(m->o, m->es));
    m->w_gateup[l] = cv.take<void*>(mat_bytes(m->gateup, m->es));
    m->w_down[l] = cv.take<void*>(mat_bytes(m->down, m->es));
    m->n1[l] = cv.take<float*>((size_t)c.d_model * 4);
    m->n2[l] = cv.take<float*>((size_t)c.d_model * 4);
  }
  m->norm_f = cv.take<float*>((size_t)c.d_model * 4);
  m->lm_head = cv.take<void*>(mat_bytes(m->lm, m->es));
  return align_up(cv.off, kAlign);
}

size_t cache_layout(rv_cache* c, void* buf) {
  const rv_config& mc = c->m->cfg;
  const int es = c->m->es, d = mc.d_model, hd = mc.head_dim;
  const int qd = mc.n_heads * hd;
  c->rows_cap = cache_rows_cap(c->B, c->max_block);
  c->out_rows_cap = round_up(c->B * 2 * (c->max_drafts + 1), 64);
  c->r1_cap = c->B * (c->max_drafts + 1);
  c->nchunk = (mc.vocab + kVocabChunk - 1) / kVocabChunk;
  c->kv_len = round_up(c->max_len, 64);
  c->kv_layer_elems = (size_t)c->B * mc.n_kv_heads * c->kv_len * hd;
  c->part_entries = cache_part_entries(c->rows_cap, mc.n_heads);
  const int nseg_cap = std::max(c->B, (int)RV_MAX_SEGS);
  Carve cv(buf);
  // bf16 models keep K and V as hi/lo bf16 planes (the operand form)
  const size_t kv_plane = c->kv_layer_elems * mc.n_layers * es, kv_lo = es == 2 ? kv_plane : 0;
  c->kc = cv.take<char*>(kv_plane);
  c->vc = cv.take<char*>(kv_plane);
  c->kc2 = cv.take<char*>(kv_lo);
  c->vc2 = cv.take<char*>(kv_lo);
  c->ids = cv.take<int*>((size_t)c->B * c->max_len * 4);
  c->rope_cos = cv.take<float*>((size_t)c->max_len * (hd / 2) * 4);
  c->rope_sin = cv.take<float*>((size_t)c->max_len * (hd / 2) * 4);
  c->seq_bad = cv.take<int*>((size_t)c->B * 4);
  c->row_pos = cv.take<int*>((size_t)c->rows_cap * 4);
  c->row_seq = cv.take<int*>((size_t)c->rows_cap * 4);
  c->row_bad = cv.take<int*>((size_t)c->rows_cap * 4);
  c->seg_b = cv.take<int*>((size_t)nseg_cap * 4);
  c->seg_row0 = cv.take<int*>((size_t)nseg_cap * 4);
  c->seg_n = cv.take<int*>((size_t)nseg_cap * 4);
  c->seg_pos0 = cv.take<int*>((size_t)nseg_cap * 4);
  c->h = cv.take<float*>((size_t)c->rows_cap * d * 4);
  // operand planes: bf16 models keep hi and lo planes of 2 bytes each,
  // fp32 models one 4-byte plane
  const size_t e1 = es == 2 ? 2 : 4, e2 = es == 2 ? 2 : 0;
  c->xn = cv.take<void*>((size_t)c->rows_cap * d * e1);
  c->xn2 = cv.take<void*>((size_t)c->rows_cap * d * e2);
  c->qbuf = cv.take<void*>((size_t)c->rows_cap * qd * e1);
  c->qbuf2 = cv.take<void*>((size_t)c->rows_cap * qd * e2);
  c->att = cv.take<void*>((size_t)c->rows_cap * qd * e1);
  c->att2 = cv.take<void*>((size_t)c->rows_cap * qd * e2);
  c->act = cv.take<void*>((size_t)c->rows_cap * mc.ffn_dim * e1);
  c->act2 = cv.take<void*>((size_t)c->rows_cap * mc.ffn_dim * e2);
  c->lm_x = cv.take<void*>((size_t)c->out_rows_cap * d * e1);
  c->lm_x2 = cv.take<void*>((size_t)c->out_rows_cap * d * e2);
  c->part_o = cv.take<float*>(c->part_entries * hd * 4);
  c->part_ml = cv.take<float*>(c->part_entries * 2 * 4);
  c->gpart_rows = std::max(kMaxSplitK * kSplitRows, kMaxSplitTiled * round_up(c->B * c->max_block, 64));
  c->gpart = cv.take<float*>((size_t)c->gpart_rows * std::max(d, c->m->qkv.N) * 4);
  c->logits = cv.take<float*>((size_t)c->out_rows_cap * mc.vocab * 4);
  c->z = cv.take<float*>((size_t)c->r1_cap * mc.vocab * 4);
  c->lp = cv.take<float*>((size_t)3 * c->r1_cap * mc.vocab * 4);
  c->hpart = cv.take<float*>((size_t)4 * c->r1_cap * c->nchunk * 4 * 4);
  c->lse = cv.take<float*>((size_t)3 * c->r1_cap * 4);
  c->margins = cv.take<float*>((size_t)c->B * (c->max_drafts + 2) * 4);
  c->entropy = cv.take<float*>((size_t)2 * c->r1_cap * 4);
  c->lm_src = cv.take<int*>((size_t)c->out_rows_cap * 4);
  c->argmax = cv.take<int*>((size_t)c->r1_cap * 4);
  return align_up(cv.off, kAlign);
}

}  // namespace
thread_local LaunchEvents g_launch_events;
namespace {

// Records a start/stop event pair around one launch when profiling is on.
// For matrix-kernel classes the pair is attached to the kernel dispatch
// itself (timestamps at kernel start and end); for the others it is recorded
// on the stream before and after the launch.
struct Prof {
  rv_cache* c;
  int cls;
  hipStream_t st;
  size_t slot = SIZE_MAX;
  bool attached = false;
  static bool is_matrix(int k) {
    return k == RV_PROF_QKV || k == RV_PROF_O || k == RV_PROF_GATEUP || k == RV_PROF_DOWN || k == RV_PROF_LMHEAD;
  }
  Prof(rv_cache* c_, int cls_, hipStream_t st_) : c(c_), cls(cls_), st(st_) {
    if (!c->prof) return;
    if (c->prof_used == c->prof_cls.size()) {
      hipEvent_t a, b;
      if (hipEventCreate(&a) != hipSuccess) return;
      if (hipEventCreate(&b) != hipSuccess) {
        (void)hipEventDestroy(a);
        return;
      }
      c->prof_ev.push_back(a);
      c->prof_ev.push_back(b);
      c->prof_cls.push_back(-1);
    }
    slot = c->prof_used++;
    c->prof_cls[slot] = cls;
    if (is_matrix(cls)) {
      attached = true;
      g_launch_events = LaunchEvents{c->prof_ev[2 * slot], c->prof_ev[2 * slot + 1]};
    } else {
      (void)hipEventRecord(c->prof_ev[2 * slot], st);
    }
  }
  ~Prof() {
    if (slot == SIZE_MAX) return;
    if (attached) {
      if (g_launch_events.start) {  // no matrix kernel consumed the pair
        (void)hipEventRecord(c->prof_ev[2 * slot], st);
        (void)hipEventRecord(c->prof_ev[2 * slot + 1], st);
        g_launch_events = LaunchEvents{};
      }
    } else {
      (void)hipEventRecord(c->prof_ev[2 * slot + 1], st);
    }
  }
};

// The matmul launch shape for this model's element type and epilogue
// (plan_matmul in rv_plan.h).
GemmPlan plan_gemm(int dtype, int epi, int M, int N, int K, bool allow_split, int part_rows) {
  return plan_matmul(dtype == RV_BF16, epi == EPI_SWIGLU, M, N, K, allow_split, part_rows);
}

hipError_t run_gemm(const rv_cache* c, int epi, GemmArgs g, bool allow_split, hipStream_t st,
                    int* gk_out = nullptr) {
  const int dtype = c->m->cfg.dtype;
  const GemmPlan p = plan_gemm(dtype, epi, g.M, g.N, g.K, allow_split, c->gpart_rows);
  g.n_tg = p.n_tg;
  g.gk = p.gk;
  if (gk_out) *gk_out = p.gk;
  const int e = (epi == EPI_RESID && p.gk > 1) ? EPI_PARTIAL : epi;
  if (p.tiled) return launch_gemm_tiled(e, g, p.nw, p.nt, p.mtt, st);
  return launch_gemm(dtype, e, g, p.nt, p.mtt, st);
}

// Runs every decoder layer over the current row plan (h filled, segments set).
// qmax: queries per (segment, kv head); kmax: 1 + largest position in the plan.
// With split_last the last down projection may leave k-group partials in
// c->gpart; *pending_out then gives their count (the final norm adds them).
rv_status run_layers(rv_cache* c, int M, int nseg, int max_seg_rows, int kmax, const int* h_seg_end,
                     const int* h_seg_rows, bool split_last, int* pending_out, hipStream_t st) {
  rv_model* m = c->m;
  const rv_config& mc = m->cfg;
  const int dt = mc.dtype, d = mc.d_model, hd = mc.head_dim;
  const int G = mc.n_heads / mc.n_kv_heads;
  const int qmax = G * max_seg_rows;
  const int groups = nseg * mc.n_kv_heads;
  const int qpw = plan_attn_queries(dt == RV_BF16, qmax);
  const int qgroups = (qmax + qpw - 1) / qpw;
  // Key split (plan_attn_split; 70B batch 8 at 8K context: 4 splits, 768
  // workgroups, 348 us per layer vs 393 us with 3 splits and 576).
  const int ks = plan_attn_split(kmax, nseg, h_seg_end, h_seg_rows, mc.n_kv_heads, G, qmax, c->part_entries, qpw);
  if (ks == 0) return rv_fail(RV_E_CAPACITY, "attention partial buffer too small for %d keys", kmax);
  const int nsplit = (kmax + ks - 1) / ks;

  AttnArgs at{};
  at.q = c->qbuf;
  at.q2 = c->qbuf2;
  at.seg_b = c->seg_b;
  at.seg_row0 = c->seg_row0;
  at.seg_n = c->seg_n;
  at.seg_pos0 = c->seg_pos0;
  at.nseg = nseg;
  at.n_heads = mc.n_heads;
  at.n_kv = mc.n_kv_heads;
  at.hd = hd;
  at.kv_len = c->kv_len;
  at.ks = ks;
  at.nsplit = nsplit;
  at.qmax = qmax;
  at.part_o = c->part_o;
  at.part_ml = c->part_ml;
  at.out = c->att;
  at.out2 = c->att2;
  at.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)hd));

  int pending = 0;  // k-groups of the last residual matmul still in c->gpart
  for (int l = 0; l < mc.n_layers; ++l) {
    const size_t lo = (size_t)l * c->kv_layer_elems * m->es;
    char* kc = c->kc + lo;
    char* vc = c->vc + lo;
    char* kc2 = m->es == 2 ? c->kc2 + lo : nullptr;
    char* vc2 = m->es == 2 ? c->vc2 + lo : nullptr;
    {
      Prof pf(c, RV_PROF_NORM, st);
      HIP_TRY(launch_rmsnorm(dt, c->h, M, d, m->n1[l], mc.rms_eps, c->xn, c->xn2, nullptr,
                             pending > 1 ? c->gpart : nullptr, pending, M, st),
              "rmsnorm");
    }

    GemmArgs g{};
    g.W = m->w_qkv[l];
    g.X = c->xn;
    g.X2 = c->xn2;
    g.M = M;
    g.N = m->qkv.N;
    g.K = d;
    g.qbuf = c->qbuf;
    g.qbuf2 = c->qbuf2;
    g.kc = kc;
    g.vc = vc;
    g.kc2 = kc2;
    g.vc2 = vc2;
    g.row_pos = c->row_pos;
    g.row_seq = c->row_seq;
    g.rope_cos = c->rope_cos;
    g.rope_sin = c->rope_sin;
    g.hd = hd;
    g.n_heads = mc.n_heads;
    g.n_kv = mc.n_kv_heads;
    g.kv_len = c->kv_len;
    g.q_rows = m->qkv.q_rows;
    g.k_rows = m->qkv.k_rows;
    {
      // few-row passes split K; the partials are finished (sum, rotary,
      // q operand and KV writes) by a small per-token kernel.  (Finishing
      // them in the last-arriving k-group workgroup instead needs an
      // agent-scope release per workgroup, an L2 writeback each: measured
      // slower than the extra launch.)
      Prof pf(c, RV_PROF_QKV, st);
      const GemmPlan qp = plan_gemm(dt, EPI_RESID, M, g.N, g.K, true, c->gpart_rows);
      if (qp.gk > 1) {
        g.P = c->gpart;
        g.ldy = g.N;
        int gk = 1;
        HIP_TRY(run_gemm(c, EPI_RESID, g, true, st, &gk), "qkv");
        QkvFinish qf{c->gpart, gk, M, g.N, g.q_rows, g.k_rows, hd, mc.n_heads, mc.n_kv_heads, c->kv_len,
                     c->row_pos, c->row_seq, c->rope_cos, c->rope_sin, c->qbuf, c->qbuf2, kc, vc, kc2, vc2};
        HIP_TRY(launch_qkv_finish(dt, qf, st), "qkv finish");
      } else {
        HIP_TRY(run_gemm(c, EPI_QKV, g, false, st), "qkv");
      }
    }

    at.kc = kc;
    at.vc = vc;
    at.kc2 = kc2;
    at.vc2 = vc2;
    {
      Prof pf(c, RV_PROF_ATTN, st);
      HIP_TRY(launch_attention(dt, at, qgroups, qpw, st), "attention");
    }
    {
      Prof pf(c, RV_PROF_COMBINE, st);
      HIP_TRY(launch_attn_combine(dt, at, st), "attention combine");
    }

    GemmArgs go{};
    go.W = m->w_o[l];
    go.X = c->att;
    go.X2 = c->att2;
    go.M = M;
    go.N = d;
    go.K = mc.n_heads * hd;
    go.Y = c->h;
    go.ldy = d;
    go.P = c->gpart;
    {
      Prof pf(c, RV_PROF_O, st);
      HIP_TRY(run_gemm(c, EPI_RESID, go, true, st, &pending), "o-proj");
    }

    {
      Prof pf(c, RV_PROF_NORM, st);
      HIP_TRY(launch_rmsnorm(dt, c->h, M, d, m->n2[l], mc.rms_eps, c->xn, c->xn2, nullptr,
                             pending > 1 ? c->gpart : nullptr, pending, M, st),
              "rmsnorm");
    }
    GemmArgs gu{};
    gu.W = m->w_gateup[l];
    gu.X = c->xn;
    gu.X2 = c->xn2;
    gu.M = M;
    gu.N = m->gateup.N;
    gu.K = d;
    gu.act = c->act;
    gu.act2 = c->act2;
    gu.ld_act = mc.ffn_dim;
    {
      Prof pf(c, RV_PROF_GATEUP, st);
      HIP_TRY(run_gemm(c, EPI_SWIGLU, gu, false, st), "gate/up");
    }

    GemmArgs gd{};
    gd.W = m->w_down[l];
    gd.X = c->act;
    gd.X2 = c->act2;
    gd.M = M;
    gd.N = d;
    gd.K = mc.ffn_dim;
    gd.Y = c->h;
    gd.ldy = d;
    gd.P = c->gpart;
    {
      Prof pf(c, RV_PROF_DOWN, st);
      HIP_TRY(run_gemm(c, EPI_RESID, gd, split_last || l + 1 < mc.n_layers, st, &pending), "down");
    }
  }
  if (pending_out) *pending_out = pending;
  return RV_OK;
}

// Physical row of a logical row of a fused matrix (inverse of mat_logical_row).
int physical_row(const MatDesc& md, int lr) {
  if (md.kind == MAT_GATEUP) {
    const int half = md.N / 2, part = lr >= half, r = lr - part * half;
    return (2 * (r / 16) + part) * 16 + r % 16;
  }
  if (md.kind == MAT_QKV && lr < md.q_rows + md.k_rows) {
    const int head = lr / md.hd, dim = lr % md.hd, hh = md.hd / 2;
    const int within = dim < hh ? 16 * (dim / 8) + dim % 8 : 16 * ((dim - hh) / 8) + 8 + (dim - hh) % 8;
    return head * md.hd + within;
  }
  return lr;
}

}  // namespace

// ======================================================================= C ABI

extern "C" {

const char* rv_status_str(rv_status s) {
  switch (s) {
    case RV_OK: return "ok";
    case RV_E_ARG: return "invalid argument";
    case RV_E_RANGE: return "prefix length out of range";
    case RV_E_CAPACITY: return "block does not fit the cache";
    case RV_E_BUFFER: return "buffer too small";
    case RV_E_HIP: return "HIP runtime error";
    case RV_E_STATE: return "invalid state";
  }
  return "unknown status";
}

const char* rv_last_error(void) { return g_err.c_str(); }

rv_status rv_model_bytes(const rv_config* cfg, size_t* bytes) {
  rv_status s = check_config(cfg);
  if (s != RV_OK) return s;
  if (!bytes) return rv_fail(RV_E_ARG, "bytes is NULL");
  rv_model m{};
  m.cfg = *cfg;
  m.es = cfg->dtype == RV_BF16 ? 2 : 4;
  describe(&m);
  *bytes = model_layout(&m, nullptr);
  return RV_OK;
}

rv_status rv_init_weights(const rv_config* cfg, uint64_t seed, void* d_buf, size_t buf_bytes, void* stream,
                          rv_model** out) {
  rv_status s = check_config(cfg);
  if (s != RV_OK) return s;
  if (!d_buf || !out) return rv_fail(RV_E_ARG, "d_buf and out must not be NULL");
  rv_model* m = new rv_model();
  m->cfg = *cfg;
  m->seed = seed;
  m->es = cfg->dtype == RV_BF16 ? 2 : 4;
  describe(m);
  size_t need = model_layout(m, nullptr);
  if (buf_bytes < need) {
    delete m;
    return rv_fail(RV_E_BUFFER, "model buffer has %zu bytes, needs %zu", buf_bytes, need);
  }
  m->base = (char*)d_buf;
  m->bytes = need;
  model_layout(m, d_buf);
  hipStream_t st = (hipStream_t)stream;
  const uint64_t seed_mix = splitmix_finalise(seed + 0x9E3779B97F4A7C15ULL);
  const float scale = (float)((double)cfg->init_std / std::sqrt(4.0 * (65536.0 * 65536.0 - 1.0) / 12.0));
  const rv_config& c = *cfg;
  const int dt = c.dtype;
  auto launch_all = [&]() -> hipError_t {
    hipError_t e = launch_init_rowmajor(dt, m->embed, 0, (size_t)c.vocab * c.d_model, seed_mix, scale, st);
    if (e != hipSuccess) return e;
    for (int l = 0; l < c.n_layers; ++l) {
      const uint64_t t = 1 + 7 * (uint64_t)l;
      const int qd = m->qkv.q_rows, kvd = m->qkv.k_rows;
      if ((e = launch_init_packed(dt, m->w_qkv[l], m->qkv, t + 0, t + 1, t + 2, qd, qd + kvd, seed_mix, scale, st)))
        return e;
      if ((e = launch_init_packed(dt, m->w_o[l], m->o, t + 3, 0, 0, 1 << 30, 1 << 30, seed_mix, scale, st))) return e;
      if ((e = launch_init_packed(dt, m->w_gateup[l], m->gateup, t + 4, t + 5, 0, c.ffn_dim, 1 << 30, seed_mix,
                                  scale, st)))
        return e;
      if ((e = launch_init_packed(dt, m->w_down[l], m->down, t + 6, 0, 0, 1 << 30, 1 << 30, seed_mix, scale, st)))
        return e;
      if ((e = launch_fill_f32(m->n1[l], 1.0f, c.d_model, st))) return e;
      if ((e = launch_fill_f32(m->n2[l], 1.0f, c.d_model, st))) return e;
    }
    if ((e = launch_fill_f32(m->norm_f, 1.0f, c.d_model, st))) return e;
    return launch_init_packed(dt, m->lm_head, m->lm, 1 + 7 * (uint64_t)c.n_layers, 0, 0, 1 << 30, 1 << 30, seed_mix,
                              scale, st);
  };
  hipError_t e = launch_all();
  if (e != hipSuccess) {
    delete m;
    return hip_fail(e, "weight init");
  }
  *out = m;
  return RV_OK;
}

void rv_model_free(rv_model* m) { delete m; }

rv_status rv_cache_bytes(const rv_model* m, int32_t batch, int32_t max_len, int32_t max_block, int32_t max_drafts,
                         size_t* bytes) {
  if (!m || !bytes) return rv_fail(RV_E_ARG, "model and bytes must not be NULL");
  if (batch <= 0 || batch > RV_MAX_BATCH) return rv_fail(RV_E_ARG, "batch must be in [1, %d]", RV_MAX_BATCH);
  if (max_len <= 0 || max_block <= 0 || max_drafts < 0 || max_drafts > RV_MAX_DRAFTS)
    return rv_fail(RV_E_ARG, "max_len, max_block must be > 0 and max_drafts in [0, %d]", RV_MAX_DRAFTS);
  rv_cache c{};
  c.m = const_cast<rv_model*>(m);
  c.B = batch;
  c.max_len = max_len;
  c.max_block = max_block;
  c.max_drafts = max_drafts;
  *bytes = cache_layout(&c, nullptr);
  return RV_OK;
}

rv_status rv_cache_create(rv_model* m, int32_t batch, int32_t max_len, int32_t max_block, int32_t max_drafts,
                          void* d_buf, size_t buf_bytes, rv_cache** out) {
  size_t need = 0;
  rv_status s = rv_cache_bytes(m, batch, max_len, max_block, max_drafts, &need);
  if (s != RV_OK) return s;
  if (!d_buf || !out) return rv_fail(RV_E_ARG, "d_buf and out must not be NULL");
  if (buf_bytes < need) return rv_fail(RV_E_BUFFER, "cache buffer has %zu bytes, needs %zu", buf_bytes, need);
  rv_cache* c = new rv_cache();
  c->m = m;
  c->B = batch;
  c->max_len = max_len;
  c->max_block = max_block;
  c->max_drafts = max_drafts;
  c->base = (char*)d_buf;
  c->bytes = need;
  cache_layout(c, d_buf);
  // rotary table: angle p * base^(-2i/hd) in fp64, stored as fp32
  const int hh = m->cfg.head_dim / 2;
  std::vector<float> cs((size_t)max_len * hh), sn((size_t)max_len * hh);
  for (int p = 0; p < max_len; ++p)
    for (int i = 0; i < hh; ++i) {
      const double theta = std::pow((double)m->cfg.rope_base, -2.0 * i / m->cfg.head_dim);
      const double ang = (double)p * theta;
      cs[(size_t)p * hh + i] = (float)std::cos(ang);
      sn[(size_t)p * hh + i] = (float)std::sin(ang);
    }
  hipError_t e = hipMemset(d_buf, 0, need);
  if (e == hipSuccess) e = hipMemcpy(c->rope_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(c->rope_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    delete c;
    return hip_fail(e, "cache setup");
  }
  *out = c;
  return RV_OK;
}

void rv_cache_free(rv_cache* c) { delete c; }

rv_status rv_prefill_cache(rv_cache* c, const int32_t* d_prefix_ids, int32_t ld, const int32_t* h_prefix_len,
                           void* stream) {
  if (!c || !d_prefix_ids || !h_prefix_len) return rv_fail(RV_E_ARG, "cache, ids and lengths must not be NULL");
  if (ld <= 0) return rv_fail(RV_E_ARG, "ld must be positive");
  for (int b = 0; b < c->B; ++b) {
    const int L = h_prefix_len[b];
    if (L < 1 || L > c->max_len || L > ld)
      return rv_fail(RV_E_RANGE, "prefix_len[%d] = %d outside [1, min(max_len=%d, ld=%d)]", b, L, c->max_len, ld);
  }
  hipStream_t st = (hipStream_t)stream;
  const rv_config& mc = c->m->cfg;
  StoreIds si{};
  si.B = c->B;
  si.ld = ld;
  si.V = mc.vocab;
  si.max_len = c->max_len;
  si.prefix = d_prefix_ids;
  si.ids = c->ids;
  si.seq_bad = c->seq_bad;
  for (int b = 0; b < c->B; ++b) si.L[b] = h_prefix_len[b];
  HIP_TRY(launch_store_ids(si, st), "store ids");

  // Chunks of up to rows_cap rows over all (sequence, position < L-1).
  PlanPrefill pp{};
  pp.ld = ld;
  pp.d = mc.d_model;
  pp.V = mc.vocab;
  pp.prefix = d_prefix_ids;
  pp.embed = c->m->embed;
  pp.h = c->h;
  pp.row_pos = c->row_pos;
  pp.row_seq = c->row_seq;
  pp.seg_b = c->seg_b;
  pp.seg_row0 = c->seg_row0;
  pp.seg_n = c->seg_n;
  pp.seg_pos0 = c->seg_pos0;
  int b = 0, pos = 0;
  PrefillChunk ch;
  while (next_prefill_chunk(h_prefix_len, c->B, c->rows_cap, b, pos, ch)) {
    pp.nseg = ch.nseg;
    pp.rows = ch.rows;
    std::copy(ch.sb, ch.sb + ch.nseg, pp.sb);
    std::copy(ch.spos0, ch.spos0 + ch.nseg, pp.spos0);
    std::copy(ch.sn, ch.sn + ch.nseg, pp.sn);
    std::copy(ch.srow0, ch.srow0 + ch.nseg, pp.srow0);
    {
      Prof pf(c, RV_PROF_PLAN, st);
      HIP_TRY(launch_plan_prefill(mc.dtype, pp, st), "prefill plan");
    }
    int seg_end[RV_MAX_SEGS];
    for (int i = 0; i < ch.nseg; ++i) seg_end[i] = ch.spos0[i] + ch.sn[i];
    rv_status s = run_layers(c, ch.rows, ch.nseg, ch.max_n, ch.kmax, seg_end, ch.sn, false, nullptr, st);
    if (s != RV_OK) return s;
  }
  c->last_k = -1;
  return RV_OK;
}

}  // extern "C"

namespace {

// Arguments of the fusion / log-softmax / accept kernels over the cache's
// logit rows (sequence b: its k_b+1 original rows, then its k_b+1 reflective
// rows).  row_bad / seq_bad are left NULL (no block: draft ids are checked).
HeadArgs head_args(rv_cache* c, int k, const uint8_t* kb, int R1, int n_probe, int P, const rv_fusion& fu,
                   const float* d_q, uint64_t seed, const int32_t* d_draft_ids, const int32_t* h_prefix_len,
                   int32_t* d_accept_len, int32_t* d_next_id) {
  HeadArgs ha{};
  ha.B = c->B;
  ha.k = k;
  ha.V = c->m->cfg.vocab;
  ha.n_probe = n_probe;
  ha.P = P;
  ha.R1 = R1;
  for (int b = 0; b < c->B; ++b) ha.kb[b] = kb[b];
  ha.max_len = c->max_len;
  ha.nchunk = c->nchunk;
  ha.chunk = kVocabChunk;
  ha.alpha = fu.alpha;
  ha.rule = fu.rule;
  ha.eps = fu.epsilon;
  ha.delta = fu.delta;
  ha.ent_src = fu.entropy_src;
  ha.temp = fu.temperature;
  ha.q = d_q;
  ha.seed = seed;
  ha.entropy = c->entropy;
  ha.logits = c->logits;
  ha.z = c->z;
  ha.part = c->hpart;
  ha.lse = c->lse;
  ha.lp = c->lp;
  ha.margins = c->margins;
  ha.drafts = d_draft_ids;
  ha.ids = c->ids;
  ha.accept_len = d_accept_len;
  ha.next_id = d_next_id;
  ha.argmax = c->argmax;
  for (int b = 0; b < c->B; ++b) ha.L[b] = h_prefix_len[b];
  return ha;
}

}  // namespace

rv_status rv_check_fusion(const rv_fusion* fusion) {
  if (!(fusion->temperature > 0.f && fusion->temperature < INFINITY))
    return rv_fail(RV_E_ARG, "temperature must be > 0 and finite");
  if (!(fusion->alpha >= 0.f && fusion->alpha <= 1.f)) return rv_fail(RV_E_ARG, "alpha must be in [0, 1]");
  if (fusion->prefix_pos < 0) return rv_fail(RV_E_ARG, "prefix_pos must be >= 0");
  if (fusion->rule != RV_RULE_GREEDY && fusion->rule != RV_RULE_TYPICAL && fusion->rule != RV_RULE_SAMPLING)
    return rv_fail(RV_E_ARG, "unknown verification rule %d", fusion->rule);
  if (fusion->rule == RV_RULE_TYPICAL) {
    if (!(fusion->epsilon > 0.f)) return rv_fail(RV_E_ARG, "epsilon must be > 0");
    if (!(fusion->delta >= 0.f)) return rv_fail(RV_E_ARG, "delta must be >= 0");
    if (fusion->entropy_src != RV_ENTROPY_FUSED && fusion->entropy_src != RV_ENTROPY_ORIGINAL)
      return rv_fail(RV_E_ARG, "unknown entropy source %d", fusion->entropy_src);
  }
  return RV_OK;
}

namespace {

// rv_verify and rv_verify_sampled: d_q / seed are used by the sampling rule only.
// k is the draft-id stride and largest draft count; h_draft_len (may be NULL:
// every sequence has k drafts) gives per-sequence counts.
rv_status verify_impl(rv_cache* c, const int32_t* h_prefix_len, const int32_t* d_draft_ids, int32_t k,
                      const int32_t* h_draft_len, const float* d_q, const int32_t* d_probe_ids, int32_t n_probe,
                      const rv_fusion* fusion, uint64_t seed, bool sampled, int32_t* d_accept_len,
                      int32_t* d_next_id, void* stream) {
  if (!c || !h_prefix_len || !fusion || !d_accept_len || !d_next_id)
    return rv_fail(RV_E_ARG, "cache, prefix_len, fusion and outputs must not be NULL");
  if (sampled != (fusion->rule == RV_RULE_SAMPLING))
    return rv_fail(RV_E_ARG, sampled ? "rv_verify_sampled needs rule RV_RULE_SAMPLING"
                                  : "the sampling rule needs the draft distributions (rv_verify_sampled)");
  if (sampled && k > 0 && !d_q) return rv_fail(RV_E_ARG, "draft distributions are NULL");
  if (k < 0 || k > c->max_drafts) return rv_fail(RV_E_ARG, "k = %d outside [0, max_drafts=%d]", k, c->max_drafts);
  if (k > 0 && !d_draft_ids) return rv_fail(RV_E_ARG, "draft ids are NULL");
  if (n_probe < 0) return rv_fail(RV_E_ARG, "n_probe must be >= 0");
  if (n_probe > 0 && !d_probe_ids) return rv_fail(RV_E_ARG, "probe ids are NULL");
  if (rv_status fs = rv_check_fusion(fusion); fs != RV_OK) return fs;
  const int P = fusion->prefix_pos;
  uint8_t kb[RV_MAX_BATCH];
  int seg_end[RV_MAX_BATCH], seg_rows[RV_MAX_BATCH];
  int S_max = 0, M = 0, R1 = 0, kmax = 0;
  for (int b = 0; b < c->B; ++b) {
    const int kk = h_draft_len ? h_draft_len[b] : k;
    if (kk < 0 || kk > k) return rv_fail(RV_E_ARG, "draft count %d of sequence %d outside [0, %d]", kk, b, k);
    kb[b] = (uint8_t)kk;
    const long long S = 1LL + 2LL * kk + n_probe + P;
    if (S > c->max_block) return rv_fail(RV_E_CAPACITY, "block of %lld rows exceeds max_block=%d", S, c->max_block);
    const int L = h_prefix_len[b];
    if (L < std::max(1, P) || L > c->max_len)
      return rv_fail(RV_E_RANGE, "prefix_len[%d] = %d outside [max(1, P)=%d, max_len=%d]", b, L, std::max(1, P),
                  c->max_len);
    if ((long long)L - 1 + S > c->max_len || (long long)L + kk + 1 > c->max_len)
      return rv_fail(RV_E_CAPACITY, "sequence %d: block of %lld rows at length %d exceeds max_len=%d", b, S, L,
                  c->max_len);
    kmax = std::max(kmax, (int)(L - 1 + S));
    seg_end[b] = (int)(L - 1 + S);
    seg_rows[b] = (int)S;
    S_max = std::max(S_max, (int)S);
    M += (int)S;
    R1 += kk + 1;
  }
  hipStream_t st = (hipStream_t)stream;
  rv_model* m = c->m;
  const rv_config& mc = m->cfg;
  const int dt = mc.dtype;

  PlanVerify pv{};
  pv.B = c->B;
  pv.S = S_max;
  pv.k = k;
  pv.lm_src = c->lm_src;
  for (int b = 0; b < c->B; ++b) pv.kb[b] = kb[b];
  pv.n_probe = n_probe;
  pv.P = P;
  pv.d = mc.d_model;
  pv.V = mc.vocab;
  pv.max_len = c->max_len;
  pv.ids = c->ids;
  pv.drafts = d_draft_ids;
  pv.probe = d_probe_ids;
  pv.embed = m->embed;
  pv.h = c->h;
  pv.row_pos = c->row_pos;
  pv.row_seq = c->row_seq;
  pv.row_bad = c->row_bad;
  pv.seg_b = c->seg_b;
  pv.seg_row0 = c->seg_row0;
  pv.seg_n = c->seg_n;
  pv.seg_pos0 = c->seg_pos0;
  for (int b = 0; b < c->B; ++b) pv.L[b] = h_prefix_len[b];
  {
    Prof pf(c, RV_PROF_PLAN, st);
    HIP_TRY(launch_plan_verify(dt, pv, st), "verify plan");
  }

  int pending = 0;
  rv_status s = run_layers(c, M, c->B, S_max, kmax, seg_end, seg_rows, true, &pending, st);
  if (s != RV_OK) return s;

  // LM head on the 2(k_b+1) rows per sequence that Algorithm 1 reads.
  const int nout = 2 * R1;
  {
    Prof pf(c, RV_PROF_NORM, st);
    HIP_TRY(launch_rmsnorm(dt, c->h, nout, mc.d_model, m->norm_f, mc.rms_eps, c->lm_x, c->lm_x2, c->lm_src,
                           pending > 1 ? c->gpart : nullptr, pending, M, st),
            "final norm");
  }
  GemmArgs gl{};
  gl.W = m->lm_head;
  gl.X = c->lm_x;
  gl.X2 = c->lm_x2;
  gl.M = nout;
  gl.N = mc.vocab;
  gl.K = mc.d_model;
  gl.Y = c->logits;
  gl.ldy = mc.vocab;
  {
    Prof pf(c, RV_PROF_LMHEAD, st);
    HIP_TRY(run_gemm(c, EPI_STORE, gl, false, st), "lm head");
  }

  HeadArgs ha = head_args(c, k, kb, R1, n_probe, P, *fusion, d_q, seed, d_draft_ids, h_prefix_len, d_accept_len,
                          d_next_id);
  ha.row_bad = c->row_bad;
  ha.seq_bad = c->seq_bad;
  {
    Prof pf(c, RV_PROF_TAIL, st);
    HIP_TRY(launch_head(ha, st), "accept");
  }
  c->last_k = k;
  c->last_R1 = R1;
  for (int b = 0; b < c->B; ++b) c->last_kb[b] = kb[b];
  return RV_OK;
}

}  // namespace

extern "C" {

rv_status rv_verify(rv_cache* c, const int32_t* h_prefix_len, const int32_t* d_draft_ids, int32_t k,
                    const int32_t* d_probe_ids, int32_t n_probe, const rv_fusion* fusion, int32_t* d_accept_len,
                    int32_t* d_next_id, void* stream) {
  return verify_impl(c, h_prefix_len, d_draft_ids, k, nullptr, nullptr, d_probe_ids, n_probe, fusion, 0, false,
                     d_accept_len, d_next_id, stream);
}

rv_status rv_verify_ragged(rv_cache* c, const int32_t* h_prefix_len, const int32_t* d_draft_ids, int32_t ld_drafts,
                           const int32_t* h_draft_len, const int32_t* d_probe_ids, int32_t n_probe,
                           const rv_fusion* fusion, int32_t* d_accept_len, int32_t* d_next_id, void* stream) {
  if (!h_draft_len) return rv_fail(RV_E_ARG, "draft lengths must not be NULL");
  return verify_impl(c, h_prefix_len, d_draft_ids, ld_drafts, h_draft_len, nullptr, d_probe_ids, n_probe, fusion, 0,
                     false, d_accept_len, d_next_id, stream);
}

rv_status rv_verify_sampled(rv_cache* c, const int32_t* h_prefix_len, const int32_t* d_draft_ids, int32_t k,
                            const float* d_draft_probs, const int32_t* d_probe_ids, int32_t n_probe,
                            const rv_fusion* fusion, uint64_t seed, int32_t* d_accept_len,
                            int32_t* d_next_id, void* stream) {
  return verify_impl(c, h_prefix_len, d_draft_ids, k, nullptr, d_draft_probs, d_probe_ids, n_probe, fusion, seed,
                     true, d_accept_len, d_next_id, stream);
}

rv_status rv_debug_fuse_accept(rv_cache* c, const float* d_logits, const int32_t* h_prefix_len,
                               const int32_t* d_draft_ids, int32_t k, const rv_fusion* fusion, int32_t* d_accept_len,
                               int32_t* d_next_id, void* stream) {
  if (!c || !d_logits || !h_prefix_len || !fusion || !d_accept_len || !d_next_id)
    return rv_fail(RV_E_ARG, "cache, logits, prefix_len, fusion and outputs must not be NULL");
  if (k < 0 || k > c->max_drafts) return rv_fail(RV_E_ARG, "k = %d outside [0, max_drafts=%d]", k, c->max_drafts);
  if (k > 0 && !d_draft_ids) return rv_fail(RV_E_ARG, "draft ids are NULL");
  if (rv_status fs = rv_check_fusion(fusion); fs != RV_OK) return fs;
  if (fusion->rule == RV_RULE_SAMPLING) return rv_fail(RV_E_ARG, "the sampling rule is not available here");
  for (int b = 0; b < c->B; ++b) {
    const int L = h_prefix_len[b];
    if (L < 1 || (long long)L + k + 1 > c->max_len)
      return rv_fail(RV_E_RANGE, "prefix_len[%d] = %d: needs 1 <= L and L + k + 1 <= max_len=%d", b, L, c->max_len);
  }
  uint8_t kb[RV_MAX_BATCH];
  for (int b = 0; b < c->B; ++b) kb[b] = (uint8_t)k;
  const int R1 = c->B * (k + 1);
  hipStream_t st = (hipStream_t)stream;
  HIP_TRY(hipMemcpyAsync(c->logits, d_logits, (size_t)2 * R1 * c->m->cfg.vocab * 4, hipMemcpyDeviceToDevice, st),
          "copy logits");
  HeadArgs ha = head_args(c, k, kb, R1, 0, 0, *fusion, nullptr, 0, d_draft_ids, h_prefix_len, d_accept_len, d_next_id);
  HIP_TRY(launch_head(ha, st), "accept");
  c->last_k = k;
  c->last_R1 = R1;
  for (int b = 0; b < c->B; ++b) c->last_kb[b] = kb[b];
  return RV_OK;
}

rv_status rv_debug_output(const rv_cache* c, int32_t which, float* d_dst, size_t dst_bytes, void* stream) {
  if (!c || !d_dst) return rv_fail(RV_E_ARG, "cache and destination must not be NULL");
  if (c->last_k < 0) return rv_fail(RV_E_STATE, "no verify has run on this cache");
  if (which < RV_OUT_ORIG || which > RV_OUT_PROB_FUSED) return rv_fail(RV_E_ARG, "unknown output %d", which);
  const int k1 = c->last_k + 1;
  hipStream_t st = (hipStream_t)stream;
  if (which == RV_OUT_ENTROPY || which == RV_OUT_MARGINS) {
    const size_t n = which == RV_OUT_ENTROPY ? (size_t)2 * c->last_R1 : (size_t)c->B * (k1 + 1);
    if (dst_bytes < n * 4) return rv_fail(RV_E_BUFFER, "destination needs %zu bytes", n * 4);
    HIP_TRY(hipMemcpyAsync(d_dst, which == RV_OUT_ENTROPY ? c->entropy : c->margins, n * 4,
                           hipMemcpyDeviceToDevice, st),
            "copy");
    return RV_OK;
  }
  const size_t V = c->m->cfg.vocab, R1 = c->last_R1, bytes = R1 * V * 4;
  if (dst_bytes < bytes) return rv_fail(RV_E_BUFFER, "destination needs %zu bytes", bytes);
  if (which == RV_OUT_ORIG || which == RV_OUT_REFL) {
    // sequence b: logit rows 2 (b + K_b) .. (o rows, then r rows), fused rows b + K_b ..
    size_t zrow = 0;
    for (int b = 0; b < c->B; ++b) {
      const size_t kb1 = (size_t)c->last_kb[b] + 1;
      const float* src = c->logits + (2 * zrow + (which == RV_OUT_REFL ? kb1 : 0)) * V;
      HIP_TRY(hipMemcpyAsync(d_dst + zrow * V, src, kb1 * V * 4, hipMemcpyDeviceToDevice, st), "copy");
      zrow += kb1;
    }
  } else if (which == RV_OUT_FUSED) {
    HIP_TRY(hipMemcpyAsync(d_dst, c->z, bytes, hipMemcpyDeviceToDevice, st), "copy");
  } else if (which == RV_OUT_PROB_FUSED) {
    HIP_TRY(launch_exp(c->lp + 2 * R1 * V, d_dst, R1 * V, st), "probabilities");
  } else {
    const size_t f = which - RV_OUT_LOGP_ORIG;
    HIP_TRY(hipMemcpyAsync(d_dst, c->lp + f * R1 * V, bytes, hipMemcpyDeviceToDevice, st), "copy");
  }
  return RV_OK;
}

rv_status rv_debug_export_kv(const rv_cache* c, int32_t layer, int32_t seq, int32_t pos0, int32_t npos, void* d_k,
                             void* d_v, size_t dst_bytes, void* stream) {
  if (!c || !d_k || !d_v) return rv_fail(RV_E_ARG, "cache and destinations must not be NULL");
  const rv_config& mc = c->m->cfg;
  if (layer < 0 || layer >= mc.n_layers || seq < 0 || seq >= c->B || pos0 < 0 || npos <= 0 ||
      (long long)pos0 + npos > c->max_len)
    return rv_fail(RV_E_ARG, "layer/seq/position range outside the cache");
  const size_t es = c->m->es, hd = mc.head_dim, row = (size_t)npos * hd * es;
  const int planes = es == 2 ? 2 : 1;
  const size_t plane = row * mc.n_kv_heads;
  if (dst_bytes < plane * planes) return rv_fail(RV_E_BUFFER, "destination needs %zu bytes", plane * planes);
  const size_t blk = (size_t)layer * c->kv_layer_elems + (size_t)seq * mc.n_kv_heads * c->kv_len * hd;
  hipStream_t st = (hipStream_t)stream;
  if (es == 2) {
    // bf16 caches are stored in attention operand order: copy out row-major
    HIP_TRY(launch_export_kv((uint16_t*)c->kc + blk, (uint16_t*)c->kc2 + blk, (int)hd, mc.n_kv_heads, c->kv_len, pos0,
                             npos, false, d_k, st),
            "export");
    HIP_TRY(launch_export_kv((uint16_t*)c->vc + blk, (uint16_t*)c->vc2 + blk, (int)hd, mc.n_kv_heads, c->kv_len, pos0,
                             npos, true, d_v, st),
            "export");
    return RV_OK;
  }
  const size_t off = (blk + (size_t)pos0 * hd) * es;
  const size_t spitch = (size_t)c->kv_len * hd * es;
  HIP_TRY(hipMemcpy2DAsync(d_k, row, c->kc + off, spitch, row, mc.n_kv_heads, hipMemcpyDeviceToDevice, st), "copy");
  HIP_TRY(hipMemcpy2DAsync(d_v, row, c->vc + off, spitch, row, mc.n_kv_heads, hipMemcpyDeviceToDevice, st), "copy");
  return RV_OK;
}

rv_status rv_commit_tokens(rv_cache* c, const int32_t* h_pos, const int32_t* d_ids, void* stream) {
  if (!c || !h_pos || !d_ids) return rv_fail(RV_E_ARG, "cache, positions and ids must not be NULL");
  for (int b = 0; b < c->B; ++b)
    if (h_pos[b] >= c->max_len) return rv_fail(RV_E_RANGE, "position %d of sequence %d >= max_len", h_pos[b], b);
  for (int b = 0; b < c->B; ++b) {
    if (h_pos[b] < 0) continue;
    HIP_TRY(hipMemcpyAsync(c->ids + (size_t)b * c->max_len + h_pos[b], d_ids + b, 4, hipMemcpyDeviceToDevice,
                           (hipStream_t)stream),
            "copy");
  }
  return RV_OK;
}

rv_status rv_debug_export_ids(const rv_cache* c, int32_t seq, int32_t pos0, int32_t n, int32_t* d_dst, void* stream) {
  if (!c || !d_dst) return rv_fail(RV_E_ARG, "cache and destination must not be NULL");
  if (seq < 0 || seq >= c->B || pos0 < 0 || n <= 0 || (long long)pos0 + n > c->max_len)
    return rv_fail(RV_E_ARG, "id range outside the cache");
  HIP_TRY(hipMemcpyAsync(d_dst, c->ids + (size_t)seq * c->max_len + pos0, (size_t)n * 4, hipMemcpyDeviceToDevice,
                         (hipStream_t)stream),
          "copy");
  return RV_OK;
}

rv_status rv_debug_weight_bits(const rv_model* m, int32_t tensor, const int64_t* h_idx, int32_t n, uint32_t* h_bits) {
  if (!m || !h_idx || !h_bits || n < 0) return rv_fail(RV_E_ARG, "bad arguments");
  const rv_config& c = m->cfg;
  const int L = c.n_layers;
  if (tensor < 0 || tensor > 1 + 7 * L) return rv_fail(RV_E_ARG, "tensor %d out of range", tensor);
  const MatDesc* md = nullptr;
  const char* base = nullptr;
  int row_off = 0;
  long long in_dim = c.d_model, rows = c.vocab;
  if (tensor == 0) {
    base = (const char*)m->embed;
  } else if (tensor == 1 + 7 * L) {
    md = &m->lm;
    base = (const char*)m->lm_head;
  } else {
    const int l = (tensor - 1) / 7, j = (tensor - 1) % 7;
    const int qd = m->qkv.q_rows, kvd = m->qkv.k_rows;
    switch (j) {
      case 0: md = &m->qkv; base = (const char*)m->w_qkv[l]; row_off = 0; rows = qd; break;
      case 1: md = &m->qkv; base = (const char*)m->w_qkv[l]; row_off = qd; rows = kvd; break;
      case 2: md = &m->qkv; base = (const char*)m->w_qkv[l]; row_off = qd + kvd; rows = kvd; break;
      case 3: md = &m->o; base = (const char*)m->w_o[l]; rows = c.d_model; in_dim = qd; break;
      case 4: md = &m->gateup; base = (const char*)m->w_gateup[l]; rows = c.ffn_dim; break;
      case 5: md = &m->gateup; base = (const char*)m->w_gateup[l]; row_off = c.ffn_dim; rows = c.ffn_dim; break;
      default: md = &m->down; base = (const char*)m->w_down[l]; rows = c.d_model; in_dim = c.ffn_dim; break;
    }
  }
  for (int i = 0; i < n; ++i) {
    const long long idx = h_idx[i];
    if (idx < 0 || idx >= rows * in_dim) return rv_fail(RV_E_ARG, "index %lld out of range", idx);
    const int r = (int)(idx / in_dim), col = (int)(idx % in_dim);
    size_t off;
    if (!md) off = (size_t)idx * m->es;
    else off = mat_packed_offset(*md, physical_row(*md, r + row_off), col, m->es);
    uint32_t v = 0;
    HIP_TRY(hipMemcpy(&v, base + off, m->es, hipMemcpyDeviceToHost), "copy");
    h_bits[i] = v;
  }
  return RV_OK;
}

rv_status rv_debug_workspace(const rv_cache* c, int32_t which, int32_t rows, void* d_dst, size_t dst_bytes,
                             void* stream) {
  if (!c || !d_dst) return rv_fail(RV_E_ARG, "cache and destination must not be NULL");
  if (rows <= 0 || rows > c->rows_cap) return rv_fail(RV_E_ARG, "rows must be in [1, %d]", c->rows_cap);
  const rv_config& mc = c->m->cfg;
  const void *src, *src2 = nullptr;
  size_t width;
  const size_t es = c->m->es;
  switch (which) {
    case RV_WS_RESID: src = c->h; width = (size_t)mc.d_model * 4; break;
    case RV_WS_ATTN: src = c->att; src2 = c->att2; width = (size_t)mc.n_heads * mc.head_dim * es; break;
    case RV_WS_ACT: src = c->act; src2 = c->act2; width = (size_t)mc.ffn_dim * es; break;
    case RV_WS_QUERY: src = c->qbuf; src2 = c->qbuf2; width = (size_t)mc.n_heads * mc.head_dim * es; break;
    default: return rv_fail(RV_E_ARG, "unknown workspace buffer %d", which);
  }
  const int planes = (src2 && es == 2) ? 2 : 1;
  if (dst_bytes < width * rows * planes)
    return rv_fail(RV_E_BUFFER, "destination needs %zu bytes", width * rows * planes);
  hipStream_t st = (hipStream_t)stream;
  if (!src2) {
    HIP_TRY(hipMemcpyAsync(d_dst, src, width * rows, hipMemcpyDeviceToDevice, st), "copy");
    return RV_OK;
  }
  // operand planes are stored in tiles: convert to row-major
  const int K = (int)(width / es);
  HIP_TRY(launch_retile(mc.dtype, src, d_dst, rows, K, false, st), "untile");
  if (planes == 2) HIP_TRY(launch_retile(mc.dtype, src2, (char*)d_dst + width * rows, rows, K, false, st), "untile");
  return RV_OK;
}

rv_status rv_debug_profile(rv_cache* c, int32_t enable) {
  if (!c) return rv_fail(RV_E_ARG, "cache must not be NULL");
  c->prof = enable != 0;
  if (c->prof) c->prof_used = 0;
  return RV_OK;
}

rv_status rv_debug_profile_read(const rv_cache* c, int32_t kclass, double* total_ms, int32_t* launches) {
  if (!c || !total_ms || !launches) return rv_fail(RV_E_ARG, "arguments must not be NULL");
  if (kclass < 0 || kclass >= RV_PROF_NCLASS) return rv_fail(RV_E_ARG, "unknown kernel class %d", kclass);
  double tot = 0.0;
  int n = 0;
  for (size_t i = 0; i < c->prof_used; ++i) {
    if (c->prof_cls[i] != kclass) continue;
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, c->prof_ev[2 * i], c->prof_ev[2 * i + 1]), "event time");
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *launches = n;
  return RV_OK;
}

rv_status rv_debug_time_matrix(rv_cache* c, int32_t matrix, int32_t M, int32_t reps, void* stream, float* avg_ms) {
  if (!c || !avg_ms) return rv_fail(RV_E_ARG, "cache and avg_ms must not be NULL");
  if (M <= 0 || M > c->rows_cap || reps <= 0) return rv_fail(RV_E_ARG, "M must be in [1, %d], reps > 0", c->rows_cap);
  if (matrix != RV_MAT_O && matrix != RV_MAT_GATEUP && matrix != RV_MAT_DOWN && matrix != RV_MAT_LM_HEAD)
    return rv_fail(RV_E_ARG, "matrix %d cannot be timed", matrix);
  rv_model* m = c->m;
  const rv_config& mc = m->cfg;
  const int dt = mc.dtype, d = mc.d_model;
  hipStream_t st = (hipStream_t)stream;
  hipEvent_t e0, e1;
  HIP_TRY(hipEventCreate(&e0), "event");
  HIP_TRY(hipEventCreate(&e1), "event");
  auto launch = [&](int rep) -> hipError_t {
    const int l = rep % mc.n_layers;
    GemmArgs g{};
    g.M = M;
    switch (matrix) {
      case RV_MAT_O:
        g.W = m->w_o[l]; g.X = c->att; g.X2 = c->att2; g.N = d; g.K = mc.n_heads * mc.head_dim;
        g.Y = c->h; g.ldy = d; g.P = c->gpart;
        return run_gemm(c, EPI_RESID, g, true, st);
      case RV_MAT_GATEUP:
        g.W = m->w_gateup[l]; g.X = c->xn; g.X2 = c->xn2; g.N = m->gateup.N; g.K = d;
        g.act = c->act; g.act2 = c->act2;
        return run_gemm(c, EPI_SWIGLU, g, false, st);
      case RV_MAT_DOWN:
        g.W = m->w_down[l]; g.X = c->act; g.X2 = c->act2; g.N = d; g.K = mc.ffn_dim;
        g.Y = c->h; g.ldy = d; g.P = c->gpart;
        return run_gemm(c, EPI_RESID, g, true, st);
      default:
        g.W = m->lm_head; g.X = c->lm_x; g.X2 = c->lm_x2; g.N = mc.vocab; g.K = d;
        g.Y = c->logits; g.ldy = mc.vocab;
        return run_gemm(c, EPI_STORE, g, false, st);
    }
  };
  if (matrix == RV_MAT_LM_HEAD && M > c->out_rows_cap) return rv_fail(RV_E_ARG, "M exceeds the LM-head rows");
  HIP_TRY(launch(0), "warm-up launch");
  HIP_TRY(hipEventRecord(e0, st), "event");
  for (int r = 0; r < reps; ++r) HIP_TRY(launch(r), "timed launch");
  HIP_TRY(hipEventRecord(e1, st), "event");
  HIP_TRY(hipEventSynchronize(e1), "event sync");
  float ms = 0.f;
  HIP_TRY(hipEventElapsedTime(&ms, e0, e1), "event time");
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  *avg_ms = ms / reps;
  c->last_k = -1;  // workspace outputs no longer describe the last verify
  return RV_OK;
}

rv_status rv_debug_linear(const rv_cache* c, int32_t layer, int32_t matrix, const void* d_x, int32_t M, float* d_y,
                          size_t y_bytes, void* stream) {
  if (!c || !d_x || !d_y) return rv_fail(RV_E_ARG, "cache, x and y must not be NULL");
  const rv_model* m = c->m;
  const rv_config& mc = m->cfg;
  if (matrix != RV_MAT_LM_HEAD && (layer < 0 || layer >= mc.n_layers)) return rv_fail(RV_E_ARG, "layer out of range");
  if (M <= 0 || M > c->rows_cap) return rv_fail(RV_E_ARG, "M must be in [1, %d]", c->rows_cap);
  const MatDesc* md;
  const void* W;
  void *xbuf, *xbuf2;
  switch (matrix) {
    case RV_MAT_QKV: md = &m->qkv; W = m->w_qkv[layer]; xbuf = c->xn; xbuf2 = c->xn2; break;
    case RV_MAT_O: md = &m->o; W = m->w_o[layer]; xbuf = c->att; xbuf2 = c->att2; break;
    case RV_MAT_GATEUP: md = &m->gateup; W = m->w_gateup[layer]; xbuf = c->xn; xbuf2 = c->xn2; break;
    case RV_MAT_DOWN: md = &m->down; W = m->w_down[layer]; xbuf = c->act; xbuf2 = c->act2; break;
    case RV_MAT_LM_HEAD: md = &m->lm; W = m->lm_head; xbuf = c->xn; xbuf2 = c->xn2; break;
    default: return rv_fail(RV_E_ARG, "unknown matrix %d", matrix);
  }
  if (y_bytes < (size_t)M * md->N * 4) return rv_fail(RV_E_BUFFER, "y needs %zu bytes", (size_t)M * md->N * 4);
  hipStream_t st = (hipStream_t)stream;
  const size_t plane = (size_t)M * md->K * m->es;
  HIP_TRY(launch_retile(mc.dtype, d_x, xbuf, M, md->K, true, st), "tile");
  if (m->es == 2) HIP_TRY(launch_retile(mc.dtype, (const char*)d_x + plane, xbuf2, M, md->K, true, st), "tile");
  GemmArgs g{};
  g.W = W;
  g.X = xbuf;
  g.X2 = xbuf2;
  g.M = M;
  g.N = md->N;
  g.K = md->K;
  g.Y = d_y;
  g.ldy = md->N;
  g.md = *md;
  HIP_TRY(run_gemm(c, EPI_STORE_LOGICAL, g, false, st), "linear");
  return RV_OK;
}

}  // extern "C"
