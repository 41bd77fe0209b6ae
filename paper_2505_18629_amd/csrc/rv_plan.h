// Host-side planning of a pass: workspace row capacities, prefill chunks and
// the attention key split.  Plain integer arithmetic with no HIP types, so
// the same code also builds for the CPU alone (the host checks under tests/).
#pragma once
#include <algorithm>
#include <cstddef>

enum { RV_MAX_SEGS = 128 };   // query segments of one prefill chunk

constexpr int kPrefillRows = 2048;    // rows per prefill chunk
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

// Key split of one attention launch (a multiple of 64 keys), or 0 if none
// fits.  Minimises the estimated time: rounds of 256 workgroups (one per CU)
// x (64-key tiles per workgroup + a per-workgroup overhead of about two
// tiles), counting the workgroups that have keys (segment s has keys
// 0 .. seg_end[s]-1 and G * seg_rows[s] queries per kv head, in groups of
// 128); bounded by the partial buffer (splits x segments x kv heads x qmax
// entries) and by the combine kernel's kMaxKeySplits splits per query.
inline int plan_attn_split(int kmax, int nseg, const int* seg_end, const int* seg_rows, int n_kv, int G, int qmax,
                           size_t part_entries) {
  const int groups = nseg * n_kv;
  int ks = 0;
  double best = 0;
  for (int cand = 64; cand <= plan_round_up(kmax, 64); cand += 64) {
    const int ns = (kmax + cand - 1) / cand;
    if (ns > kMaxKeySplits || (size_t)ns * groups * qmax > part_entries) continue;
    long long wgs = 0;
    for (int s = 0; s < nseg; ++s)
      wgs += (long long)((seg_end[s] + cand - 1) / cand) * n_kv * ((G * seg_rows[s] + 127) / 128);
    const double t = (double)((wgs + 255) / 256) * (cand / 64 + 2);
    if (ks == 0 || t < best) {
      best = t;
      ks = cand;
    }
  }
  return ks;
}
