// Host-side planning of a pass: workspace row capacities, prefill chunks,
// matmul launch shapes and the attention key split.  Plain integer arithmetic with no HIP types, so
// the same code also builds for the CPU alone (the host checks under tests/).
#pragma once
#include <algorithm>
#include <cstddef>

enum { RV_MAX_SEGS = 128 };   // query segments of one prefill chunk

constexpr int kPrefillRows = 2048;    // rows per prefill chunk
constexpr int kMaxSplitK = 16;        // k-groups of a split matmul
constexpr int kMaxSplitTiled = 4;     // k-groups of a split many-token matmul
constexpr int kSplitRows = 64;        // matmuls with at most this many rows may split K
constexpr int kSplitsPerQuery = 8;    // attention partial-buffer depth per query row
constexpr int kMaxKeySplits = 64;     // key splits the combine kernel merges per query

inline int plan_round_up(int x, int a) { return (x + a - 1) / a * a; }

// Rows of the cache workspace: a verify block of every sequence, or a prefill chunk.
inline int cache_rows_cap(int batch, int max_block) {
  return plan_round_up(std::max(batch * max_block, kPrefillRows), 64);
}

// Entries (query rows x heads x splits) of the attention partial buffers.
inline size_t cache_part_entries(int rows_cap, int n_heads) {
  return (size_t)rows_cap * n_heads * kSplitsPerQuery;
}

// One prefill chunk: up to rows_cap rows over (sequence, position < L - 1),
// as up to RV_MAX_SEGS segments.  Segment i is sequence sb[i], positions
// spos0[i] .. spos0[i] + sn[i] - 1, at rows srow0[i] ..; kmax is the largest
// position + 1 and max_n the longest segment.
struct PrefillChunk {
  int nseg, rows, max_n, kmax;
  int sb[RV_MAX_SEGS], spos0[RV_MAX_SEGS], sn[RV_MAX_SEGS], srow0[RV_MAX_SEGS];
};

// Fills the next chunk starting at (sequence b, position pos) and advances
// them; false when every sequence's positions 0 .. L_b - 2 are covered.
inline bool next_prefill_chunk(const int* L, int B, int rows_cap, int& b, int& pos, PrefillChunk& ch) {
  while (b < B && pos >= L[b] - 1) {
    ++b;
    pos = 0;
  }
  if (b >= B) return false;
  ch.rows = ch.nseg = ch.max_n = ch.kmax = 0;
  while (b < B && ch.rows < rows_cap && ch.nseg < RV_MAX_SEGS) {
    const int avail = L[b] - 1 - pos;
    if (avail <= 0) {
      ++b;
      pos = 0;
      continue;
    }
    const int n = std::min(avail, rows_cap - ch.rows);
    ch.sb[ch.nseg] = b;
    ch.spos0[ch.nseg] = pos;
    ch.sn[ch.nseg] = n;
    ch.srow0[ch.nseg] = ch.rows;
    ++ch.nseg;
    ch.rows += n;
    pos += n;
    ch.max_n = std::max(ch.max_n, n);
    ch.kmax = std::max(ch.kmax, pos);
  }
  return true;
}

// Queries per workgroup of the bf16 attention kernel: 128 (8 waves of one
// 16-query tile), or 192 (12 waves) when a kv head has 129-192 queries,
// which would otherwise take a second, mostly idle group of 128 (5 query
// heads per kv head x 31 block rows = 155, e.g. the 14B shape at k = 5 with a
// 16-token probe: 4 x 2048 keys, 30.4-32.7 -> 27.5-29.0 us per launch).
inline int plan_attn_queries(bool bf16, int qmax) { return bf16 && qmax > 128 && qmax <= 192 ? 192 : 128; }

// Key split of one attention launch (a multiple of 64 keys), or 0 if none
// fits.  Minimises the estimated time: rounds of 256 workgroups (one per CU)
// x (64-key tiles per workgroup + a per-workgroup overhead of about two
// tiles), counting the workgroups that have keys (segment s has keys
// 0 .. seg_end[s]-1 and G * seg_rows[s] queries per kv head, in groups of
// qpw); bounded by the partial buffer (splits x segments x kv heads x qmax
// entries) and by the combine kernel's kMaxKeySplits splits per query.
inline int plan_attn_split(int kmax, int nseg, const int* seg_end, const int* seg_rows, int n_kv, int G, int qmax,
                           size_t part_entries, int qpw = 128) {
  const int groups = nseg * n_kv;
  int ks = 0;
  double best = 0;
  for (int cand = 64; cand <= plan_round_up(kmax, 64); cand += 64) {
    const int ns = (kmax + cand - 1) / cand;
    if (ns > kMaxKeySplits || (size_t)ns * groups * qmax > part_entries) continue;
    long long wgs = 0;
    for (int s = 0; s < nseg; ++s)
      wgs += (long long)((seg_end[s] + cand - 1) / cand) * n_kv * ((G * seg_rows[s] + qpw - 1) / qpw);
    const double t = (double)((wgs + 255) / 256) * (cand / 64 + 2);
    if (ks == 0 || t < best) {
      best = t;
      ks = cand;
    }
  }
  return ks;
}

// Launch shape of one matmul: row tiles per workgroup (nt), token tiles
// (mtt), token groups and k-groups.  Aims for >= 384 workgroups (1.5 per CU)
// with as many rows per workgroup as possible, since every workgroup reads
// its k-range of all operand tiles; K is split across workgroups only for
// residual-stream outputs of few-row passes (the next RMSNorm adds the
// partials).
struct GemmPlan {
  bool tiled;  // many-token kernel (launch_gemm_tiled)
  int nt, mtt, n_tg, gk;
  int nw;      // waves per workgroup of the many-token kernel
};

// part_rows: capacity of the partial buffer in rows (gk * M must fit);
// bf16: the element type (k-steps of 32, else 16); swiglu: gate/up tile pairs.
inline GemmPlan plan_matmul(bool bf16, bool swiglu, int M, int N, int K, bool allow_split, int part_rows) {
  constexpr int kTarget = 384;
  const int ksteps = K / (bf16 ? 32 : 16);
  GemmPlan p{};
  p.gk = 1;
  // Many tokens (bf16): the LDS-tiled kernel (one 8- or 12-wave workgroup per CU)
  // streams the weights about once for all token groups.  The shape is
  // chosen to minimise (rounds of 256 workgroups) x (work per workgroup),
  // ties broken as below (measured over the 8B, 14B and 70B matrices at
  // 172-496 tokens: within 6% of the best of every shape tried).  K is split only for outputs whose
  // consumer adds k-group partials.
  if (bf16 && M > kSplitRows && N % 256 == 0) {
    p.tiled = true;
    long long best_cost = -1, best_wgs = 0;
    // (waves, row tiles per wave, token tiles).  A workgroup's time goes as
    // its waves per SIMD times each wave's work.  Twelve waves (three per
    // SIMD, two row tiles each) give 3/4 of the 8-wave 4 x 4 workgroup's
    // work, for matrices whose 8-wave split leaves CUs idle in a single round
    // (14B gate/up at 172 tokens: 162 -> 216 workgroups); six token tiles
    // do the same for widths that twelve waves do not divide (14B QKV at
    // 172 tokens: 168 -> 224 workgroups, 39.8 -> 35.3 us).  Equal costs go
    // to fewer workgroups, then more row tiles per wave (each staged operand
    // tile feeds that many MFMAs, so 4 row tiles need half the LDS reads per
    // MFMA of 2: O and down as 4 x 4 instead of 2 x 8, 8B batch 16 17.91 ->
    // 17.76 ms, 70B 126.9 -> 124.9 ms), then more waves per workgroup (the
    // 14B gate/up: 12 waves x 4 token tiles 104 us, 8 waves x 6 token tiles
    // 108 us), then larger tiles.
    const int shapes[][3] = {{8, 4, 8}, {8, 2, 8}, {8, 4, 4}, {8, 2, 4}, {12, 2, 4}, {8, 2, 6}};
    for (const auto& sh : shapes) {
      const int nw = sh[0], nt = sh[1], mt = sh[2];
      if (N % (16 * nw * nt)) continue;
      const int n_tg = (M + 16 * mt - 1) / (16 * mt);
      for (int gk = 1; gk <= (allow_split ? kMaxSplitTiled : 1); gk *= 2) {
        if (ksteps % gk || (ksteps / gk) % 4 || (gk > 1 && gk * M > part_rows)) continue;
        const long long wgs = (long long)(N / (16 * nw * nt)) * gk * n_tg;
        if (nw == 12 && wgs > 256) continue;
        const long long cost = (wgs + 255) / 256 * nw * nt * mt * (ksteps / gk);
        const bool better = best_cost < 0 || cost < best_cost || (cost == best_cost && wgs < best_wgs) ||
                            (cost == best_cost && wgs == best_wgs && nt > p.nt) ||
                            (cost == best_cost && wgs == best_wgs && nt == p.nt && nw > p.nw) ||
                            (cost == best_cost && wgs == best_wgs && nt == p.nt && nw == p.nw && nt * mt > p.nt * p.mtt);
        if (better) {
          best_cost = cost;
          best_wgs = wgs;
          p.nw = nw;
          p.nt = nt;
          p.mtt = mt;
          p.n_tg = n_tg;
          p.gk = gk;
        }
      }
    }
    if (best_cost >= 0) return p;
    p.tiled = false;
    p.gk = 1;
  }
  p.mtt = M <= 16 ? 1 : M <= 32 ? 2 : 4;
  p.n_tg = (M + 16 * p.mtt - 1) / (16 * p.mtt);
  const int nt_min = swiglu ? 2 : 1;
  // Large bf16 matrices against two token tiles stream best with 8 row
  // tiles per workgroup: half the operand re-reads per weight byte, and
  // ~200 workgroups already saturate HBM (8B gate/up: 5.1 -> 6.0 TB/s).
  const bool wide = bf16 && p.mtt == 2 && (long long)N * K >= (32LL << 20) && N % 128 == 0;
  if (allow_split && M <= kSplitRows && N % 64 == 0) {
    // Prefer a launch of exactly one workgroup per CU (measured at the 8B
    // shapes: down 8 tiles x 8 k-groups 22.6 -> 21.4 us, QKV 6 x 4
    // 12.8 -> 11.1 us, O 4 x 4 8.3 -> 8.1 us), with 4 and 3 row tiles tried
    // before 6: the QKV then runs 3 tiles x 2 k-groups, half the partials
    // for the finish kernel to add (the 8B batch-1 pass 3.951 -> 3.944 ms;
    // O as 2 x 2 and down as 2 x 2 or 4 x 4 measured slower).
    const int nts[] = {8, 4, 3, 6, 2};
    const int cand1[] = {2, 4, 7, 8, 14, 16};
    for (int nt : nts) {
      if ((nt == 8 && !wide) || (nt > 4 && p.mtt > 2) || N % (16 * nt)) continue;
      for (int gk : cand1) {
        if (ksteps % (4 * gk) || gk * M > part_rows) continue;
        if ((long long)(N / (16 * nt)) * gk * p.n_tg == 256) {
          p.nt = nt;
          p.gk = gk;
          return p;
        }
      }
    }
    p.nt = wide ? 8 : 4;
    const int target = wide ? kTarget / 2 : kTarget;
    const int cand[] = {1, 2, 4, 7, 8, 14, 16};
    for (int gk : cand) {
      if (ksteps % (4 * gk) || gk * M > part_rows) continue;
      p.gk = gk;
      if ((long long)(N / (16 * p.nt)) * gk * p.n_tg >= target) break;
    }
    return p;
  }
  if (wide && (long long)(N / 128) * p.n_tg >= kTarget / 2) {
    p.nt = 8;
    return p;
  }
  p.nt = 4;
  while (p.nt > nt_min && (N % (16 * p.nt) || (long long)(N / (16 * p.nt)) * p.n_tg < kTarget)) p.nt /= 2;
  while (N % (16 * p.nt)) p.nt /= 2;
  return p;
}
