// CPU check of the library's host-side planning (rv_plan.h) at the shapes of
// the benchmark workloads and at edge cases: every prefill chunk stays inside
// the workspace and segment arrays and covers each sequence's positions once,
// every attention launch's key split fits the partial buffer and the grid
// limits, and every matmul launch shape is one the launchers instantiate.
// Built with the address and undefined-behaviour sanitizers by
// tests/test_host_checks.py; exits non-zero on the first violation.
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "rv_plan.h"

namespace {

int failures = 0;

#define CHECK(cond, ...)                          \
  do {                                            \
    if (!(cond)) {                                \
      std::fprintf(stderr, "FAIL %s: ", #cond);   \
      std::fprintf(stderr, __VA_ARGS__);          \
      std::fprintf(stderr, "\n");                 \
      ++failures;                                 \
      return;                                     \
    }                                             \
  } while (0)

struct Shape {
  const char* name;
  int n_heads, n_kv;
};

// One attention launch over segments (seg_end, seg_rows): the split, the
// partial-buffer entries and the grids of the attention and combine kernels.
void check_attention(const Shape& sh, int kmax, int nseg, const int* seg_end, const int* seg_rows, int max_seg_rows,
                     size_t part_entries, const char* what) {
  const int G = sh.n_heads / sh.n_kv;
  const int qmax = G * max_seg_rows;
  const int qpw = plan_attn_queries(true, qmax);
  CHECK(qpw == 128 || qpw == 192, "%s %s: %d queries per workgroup", sh.name, what, qpw);
  const int ks = plan_attn_split(kmax, nseg, seg_end, seg_rows, sh.n_kv, G, qmax, part_entries, qpw);
  CHECK(ks > 0 && ks % 64 == 0, "%s %s: no key split for kmax %d", sh.name, what, kmax);
  const long long nsplit = (kmax + ks - 1) / ks;
  CHECK(nsplit <= kMaxKeySplits, "%s %s: %lld splits", sh.name, what, nsplit);
  CHECK((size_t)nsplit * nseg * sh.n_kv * qmax <= part_entries, "%s %s: partial entries", sh.name, what);
  const long long units = nsplit * nseg * sh.n_kv;
  const long long grid = (units + 7) / 8 * 8 * ((qmax + qpw - 1) / qpw);
  CHECK(grid > 0 && grid < (1LL << 31), "%s %s: attention grid %lld", sh.name, what, grid);
  CHECK((long long)(qmax + 3) / 4 < (1LL << 31) && (long long)nseg * sh.n_kv < 65536, "%s %s: combine grid", sh.name,
        what);
  for (int s = 0; s < nseg; ++s) CHECK(seg_end[s] <= kmax, "%s %s: segment %d ends past kmax", sh.name, what, s);
}

// Prefill of `L` (one length per sequence) in a cache of B sequences with
// blocks of up to max_block rows.
void check_prefill(const Shape& sh, const std::vector<int>& L, int max_block, int max_len) {
  const int B = (int)L.size();
  const int rows_cap = cache_rows_cap(B, max_block);
  const size_t part = cache_part_entries(rows_cap, sh.n_heads);
  std::vector<long long> covered(B, 0);
  std::vector<int> next_pos(B, 0);
  int b = 0, pos = 0, chunks = 0;
  PrefillChunk ch;
  while (next_prefill_chunk(L.data(), B, rows_cap, b, pos, ch)) {
    ++chunks;
    CHECK(ch.nseg >= 1 && ch.nseg <= RV_MAX_SEGS, "%s: chunk %d has %d segments", sh.name, chunks, ch.nseg);
    CHECK(ch.rows >= 1 && ch.rows <= rows_cap, "%s: chunk %d has %d rows (cap %d)", sh.name, chunks, ch.rows, rows_cap);
    int row = 0, seg_end[RV_MAX_SEGS];
    for (int i = 0; i < ch.nseg; ++i) {
      const int s = ch.sb[i];
      CHECK(s >= 0 && s < B, "%s: segment sequence %d", sh.name, s);
      CHECK(ch.srow0[i] == row, "%s: segment rows not consecutive", sh.name);
      CHECK(ch.sn[i] >= 1 && ch.spos0[i] == next_pos[s] && ch.spos0[i] + ch.sn[i] <= L[s] - 1,
            "%s: segment %d of sequence %d covers %d..%d (L %d, next %d)", sh.name, i, s, ch.spos0[i],
            ch.spos0[i] + ch.sn[i] - 1, L[s], next_pos[s]);
      CHECK(ch.spos0[i] + ch.sn[i] <= max_len, "%s: position past max_len", sh.name);
      next_pos[s] += ch.sn[i];
      covered[s] += ch.sn[i];
      row += ch.sn[i];
      seg_end[i] = ch.spos0[i] + ch.sn[i];
      CHECK(ch.sn[i] <= ch.max_n && seg_end[i] <= ch.kmax, "%s: chunk extents", sh.name);
    }
    CHECK(row == ch.rows, "%s: rows", sh.name);
    check_attention(sh, ch.kmax, ch.nseg, seg_end, ch.sn, ch.max_n, part, "prefill");
    if (failures) return;
  }
  for (int s = 0; s < B; ++s)
    CHECK(covered[s] == std::max(L[s] - 1, 0), "%s: sequence %d covered %lld of %d", sh.name, s, covered[s], L[s] - 1);
  std::printf("%s prefill B=%d: %d chunks, rows_cap %d, partial entries %zu\n", sh.name, B, chunks, rows_cap, part);
}

// A verify pass: one segment of S rows per sequence at positions L-1 ...
void check_verify(const Shape& sh, const std::vector<int>& L, int S, int max_block) {
  const int B = (int)L.size();
  const int rows_cap = cache_rows_cap(B, max_block);
  CHECK(S <= max_block && B * S <= rows_cap, "%s: verify rows", sh.name);
  std::vector<int> seg_end(B), seg_rows(B, S);
  int kmax = 0;
  for (int b = 0; b < B; ++b) {
    seg_end[b] = L[b] - 1 + S;
    kmax = std::max(kmax, seg_end[b]);
  }
  check_attention(sh, kmax, B, seg_end.data(), seg_rows.data(), S, cache_part_entries(rows_cap, sh.n_heads), "verify");
  std::printf("%s verify B=%d S=%d: ok\n", sh.name, B, S);
}

// One matmul launch as planned: the shape must be one the launchers
// instantiate, divide N into whole row groups and K into whole k-step
// batches, fit the partial buffer and the grid limit.
void check_matmul(const char* what, bool bf16, bool swiglu, bool allow_split, int M, int N, int K, int part_rows) {
  const GemmPlan p = plan_matmul(bf16, swiglu, M, N, K, allow_split, part_rows);
  const int ksteps = K / (bf16 ? 32 : 16);
  CHECK(p.gk >= 1 && (p.gk == 1 || allow_split), "%s M=%d: k-groups %d", what, M, p.gk);
  CHECK(p.gk == 1 || (long long)p.gk * M <= part_rows, "%s M=%d: %d k-groups x %d rows past %d", what, M, p.gk, M,
        part_rows);
  if (p.tiled) {
    const bool known = (p.nw == 8 && (p.nt == 4 || p.nt == 2) && (p.mtt == 8 || p.mtt == 4)) ||
                       (p.nw == 8 && p.nt == 2 && p.mtt == 6) || (p.nw == 12 && p.nt == 2 && p.mtt == 4);
    CHECK(bf16 && known, "%s M=%d: no many-token kernel (%d waves, %d x %d)", what, M, p.nw, p.nt, p.mtt);
    CHECK(N % (16 * p.nw * p.nt) == 0, "%s M=%d: N %d not whole row groups", what, M, N);
    CHECK(ksteps % p.gk == 0 && (ksteps / p.gk) % 4 == 0, "%s M=%d: k-steps %d / %d", what, M, ksteps, p.gk);
    CHECK(p.n_tg * p.mtt * 16 >= M, "%s M=%d: token groups", what, M);
    const long long rk = (long long)(N / (16 * p.nw * p.nt)) * p.gk;
    CHECK((rk + 7) / 8 * 8 * p.n_tg < (1LL << 31), "%s M=%d: grid", what, M);
  } else {
    const bool nt_ok = p.nt == 1 || p.nt == 2 || p.nt == 4 || p.nt == 8 || ((p.nt == 3 || p.nt == 6) && p.gk > 1);
    CHECK(nt_ok && (!swiglu || (p.nt % 2 == 0)), "%s M=%d: %d row tiles", what, M, p.nt);
    CHECK((p.mtt == 1 || p.mtt == 2 || (p.mtt == 4 && p.nt <= 4)), "%s M=%d: %d token tiles with %d row tiles", what,
          M, p.mtt, p.nt);
    CHECK(N % (16 * p.nt) == 0, "%s M=%d: N %d, %d row tiles", what, M, N, p.nt);
    CHECK(ksteps % (4 * p.gk) == 0, "%s M=%d: k-steps %d, %d k-groups", what, M, ksteps, p.gk);
    CHECK(p.n_tg * p.mtt * 16 >= M, "%s M=%d: token groups", what, M);
    CHECK((long long)p.n_tg * p.gk * (N / (16 * p.nt)) < (1LL << 31), "%s M=%d: grid", what, M);
  }
}

// Every matmul of a pass over M rows (the verify block or a prefill chunk),
// and the LM head over n_out rows.
void check_matmuls(const char* name, bool bf16, int d, int hq, int hkv, int hd, int F, int V, int M, int n_out,
                   int part_rows) {
  const int n0 = failures;
  const int nqkv = (hq + 2 * hkv) * hd;
  const GemmPlan q = plan_matmul(bf16, false, M, nqkv, d, true, part_rows);
  check_matmul("qkv", bf16, false, q.gk > 1, M, nqkv, d, part_rows);
  check_matmul("o", bf16, false, true, M, d, hq * hd, part_rows);
  check_matmul("gate/up", bf16, true, false, M, 2 * F, d, part_rows);
  check_matmul("down", bf16, false, true, M, d, F, part_rows);
  check_matmul("down (last, unsplit)", bf16, false, false, M, d, F, part_rows);
  if (n_out > 0) check_matmul("lm head", bf16, false, false, n_out, V, d, part_rows);
  if (failures == n0) std::printf("%s matmuls M=%d: ok\n", name, M);
}

// The matmuls of a model's verify passes and prefill chunks at several row
// counts (full and ragged chunks, the verify block of each batch).
void check_model_matmuls(const char* name, bool bf16, int d, int hq, int hkv, int hd, int F, int V,
                         std::vector<int> verify_rows, int batch, int max_block) {
  const int part_rows = std::max(kMaxSplitK * kSplitRows, kMaxSplitTiled * plan_round_up(batch * max_block, 64));
  for (int M : verify_rows) check_matmuls(name, bf16, d, hq, hkv, hd, F, V, M, 2 * 6 * batch, part_rows);
  for (int M : {kPrefillRows, 2047, 1023, 129, 65, 64, 33, 17, 16, 1})
    check_matmuls(name, bf16, d, hq, hkv, hd, F, V, M, 0, part_rows);
}

}  // namespace

int main() {
  const Shape s8{"8b", 32, 8}, s14{"14b", 40, 8}, s70{"70b", 64, 8}, tiny{"tiny", 4, 4};
  // the benchmark workloads (prefix lengths as drawn: the ragged batch
  // spans 512..4096)
  check_prefill(tiny, {128}, 64, 160);
  check_verify(tiny, {128}, 21, 64);
  check_prefill(s8, {1024}, 64, 1100);
  check_verify(s8, {1024}, 31, 64);
  std::vector<int> ragged;
  for (int b = 0; b < 16; ++b) ragged.push_back(512 + (b * 229) % 3585);
  ragged[3] = 4096;
  ragged[7] = 512;
  check_prefill(s8, ragged, 64, 4140);
  check_verify(s8, ragged, 31, 64);
  check_prefill(s14, std::vector<int>(4, 2048), 64, 2100);
  check_verify(s14, std::vector<int>(4, 2048), 43, 64);
  check_prefill(s70, std::vector<int>(8, 8192), 64, 8245);
  check_verify(s70, std::vector<int>(8, 8192), 45, 64);
  // edge cases: nothing to prefill, the largest batch of short prefixes
  // (segment limit), one position, a block filling max_len
  check_prefill(s70, std::vector<int>(8, 1), 64, 64);
  check_prefill(s8, std::vector<int>(256, 3), 8, 64);
  check_prefill(s8, std::vector<int>(256, 300), 8, 400);
  check_verify(s8, std::vector<int>(256, 300), 8, 8);
  check_prefill(s70, {2, 8192, 1, 4097}, 128, 8400);
  check_verify(s70, {2, 8192, 1, 4097}, 128, 128);
  // matmul launch shapes: the benchmark models at their verify blocks
  // (8B batch 1 and 16, 14B batch 4, 70B batch 8) and prefill chunks, and
  // the tiny parity shapes
  check_model_matmuls("8b", true, 4096, 32, 8, 128, 14336, 128256, {31, 496, 8 * 256}, 256, 64);
  check_model_matmuls("14b", true, 5120, 40, 8, 128, 13824, 152064, {172}, 4, 64);
  check_model_matmuls("70b", true, 8192, 64, 8, 128, 28672, 128256, {248, 360}, 8, 64);
  check_model_matmuls("tiny-f32", false, 256, 4, 4, 64, 1024, 4096, {21, 84}, 4, 64);
  check_model_matmuls("tiny-gqa-bf16", true, 256, 8, 2, 32, 768, 4096, {21, 84, 130}, 8, 64);
  if (failures) {
    std::fprintf(stderr, "%d failure(s)\n", failures);
    return 1;
  }
  std::printf("all plans in bounds\n");
  return 0;
}
