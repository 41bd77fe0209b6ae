// Fusion, log-softmax and the accept decision of one verify pass.
//
//  1. k_fuse_stats   z_i = (1 - alpha) o_i + alpha r_i (Eq. 2, fp32, no FMA
//                    contraction, so alpha = 0 and alpha = 1 give o and r
//                    exactly) and, per vocabulary chunk, the max, the sum of
//                    exp and the centred sum of exp * (x - max) of o, r and
//                    z, plus z's top-2 and argmax.
//  2. k_accept       per sequence: merges the chunks in index order, gives
//                    log-sum-exp and entropy (H = log S - S1 / S for the
//                    centred sums), x_hat_i = argmax z_i (lowest id on
//                    ties), applies the exact-match rule (Algorithm 2 at
//                    temperature 0) or the entropy-thresholded rule
//                    (Algorithm 3), emits t = x_hat_{n+1} and appends
//                    x_1..x_n, t to the id history.
//                    With the sampling rule (Algorithm 1) it only decides
//                    n, from Philox4x64-10 uniforms r_i.
//  2b. k_sample, k_sample_finish   sampling rule: per vocabulary chunk the
//                    best Gumbel-perturbed score of the residual
//                    max(0, p_{n+1} - q_{n+1}) (or p_{k+1}); then per sequence
//                    the chunk maxima merged in order give t.
//  3. k_logprob      log-softmax rows of o, r and z (pass two).
#include "rv_internal.h"

#pragma clang fp contract(off)

namespace {

struct Top {
  float m1;   // max
  int i1;     // its lowest index
  float m2;   // second largest value (equal to m1 on ties)
};

RV_DEV Top top_merge(Top a, Top b) {
  if (b.m1 > a.m1 || (b.m1 == a.m1 && b.i1 < a.i1)) {
    Top t = a;
    a = b;
    b = t;
  }
  a.m2 = fmaxf(a.m2, b.m1);
  return a;
}

// Philox4x64-10 (Salmon et al., SC 2011): 10 rounds of two 64x64->128-bit
// products of counter words 0 and 2 with fixed odd constants, mixed with the
// other words and the key; the key advances by two Weyl constants between
// rounds.
RV_DEV void philox4x64(uint64_t (&c)[4], uint64_t k0, uint64_t k1) {
  constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t lo0 = M0 * c[0], hi0 = __umul64hi(M0, c[0]);
    const uint64_t lo1 = M1 * c[2], hi1 = __umul64hi(M1, c[2]);
    const uint64_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
    if (r < 9) {
      k0 += W0;
      k1 += W1;
    }
  }
}

// ((w >> 41) + 1/2) / 2^23: a uniform in (0, 1), exact in fp32.
RV_DEV float uniform23(uint64_t w) { return ((float)(w >> 41) + 0.5f) * (1.0f / 8388608.0f); }

// Sequence b of fused row r and the row's index i within it (sequence b owns
// rows b + K_b .. b + K_b + k_b).
RV_DEV void fused_row_seq(const uint8_t* kb, int B, int r, int& b, int& i) {
  int start = 0;
  for (b = 0; b < B - 1; ++b) {
    const int n = kb[b] + 1;
    if (r < start + n) break;
    start += n;
  }
  i = r - start;
}

// Softmax statistics of a set of values: max m, S = sum exp(x - m) and the
// centred S1 = sum exp(x - m) (x - m).  Empty sets have m = -inf, S = S1 = 0.
struct Stat {
  float m, s, s1;
};

RV_DEV Stat stat_merge(Stat a, Stat b) {
  const float mn = fmaxf(a.m, b.m);
  if (mn == -INFINITY) return a;
  Stat r{mn, 0.f, 0.f};
  if (a.m != -INFINITY) {
    const float d = a.m - mn, e = __expf(d);
    r.s += a.s * e;
    r.s1 += e * (a.s1 + a.s * d);
  }
  if (b.m != -INFINITY) {
    const float d = b.m - mn, e = __expf(d);
    r.s += b.s * e;
    r.s1 += e * (b.s1 + b.s * d);
  }
  return r;
}

RV_DEV Stat stat_shfl(Stat a, int off) {
  return Stat{__shfl_xor(a.m, off, 64), __shfl_xor(a.s, off, 64), __shfl_xor(a.s1, off, 64)};
}

template <int E>
RV_DEV Stat stat_of(const float (&x)[E], int n_valid) {
  float m = -INFINITY;
#pragma unroll
  for (int e = 0; e < E; ++e)
    if (e < n_valid) m = fmaxf(m, x[e]);
  Stat r{m, 0.f, 0.f};
  if (m == -INFINITY) return r;
#pragma unroll
  for (int e = 0; e < E; ++e)
    if (e < n_valid) {
      const float d = x[e] - m, p = __expf(d);
      r.s += p;
      r.s1 += p > 0.f ? p * d : 0.f;  // 0 log 0 = 0 (ids at -inf)
    }
  return r;
}

// Fused logit z_i[v] of fused row `row` whose o and r rows are lrow_o and
// lrow_r: read back from the fused rows, or, where none are kept (z NULL),
// recomputed from o and r with k_fuse_stats's own expression, which gives the
// same bits.
RV_DEV float fused_at(const HeadArgs& a, int row, int lrow_o, int lrow_r, int v) {
  if (a.z) return a.z[(size_t)row * a.V + v];
  const float zo = (1.0f - a.alpha) * a.logits[(size_t)lrow_o * a.V + v];
  const float zr = a.alpha * a.logits[(size_t)lrow_r * a.V + v];
  float z = zo + zr;
  if (a.temp != 1.0f) z = z / a.temp;
  return z;
}

// One workgroup per (vocabulary chunk of 2048, fused row); each thread owns 8
// entries, strided by 256, and loads them all before computing.
__global__ __launch_bounds__(256) void k_fuse_stats(HeadArgs a) {
  constexpr int E = 8;
  const int chunk = blockIdx.x, row = blockIdx.y;  // fused row
  int b, i;
  fused_row_seq(a.kb, a.B, row, b, i);
  const int k1 = a.kb[b] + 1, lrow0 = 2 * (row - i);  // first logit row of sequence b
  const float* o = a.logits + ((size_t)lrow0 + i) * a.V;
  const float* r = a.logits + ((size_t)lrow0 + k1 + i) * a.V;
  float* z = a.z ? a.z + (size_t)row * a.V : nullptr;  // fused rows kept for inspection
  const float wa = a.alpha, wo = 1.0f - a.alpha;
  const int v0 = chunk * a.chunk, v1 = min(a.V, v0 + a.chunk);
  float ov[E], rv[E], zv[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int v = min(v0 + threadIdx.x + e * 256, v1 - 1);
    ov[e] = o[v];
    rv[e] = r[v];
  }
  // entries e < n_valid are inside the chunk (v increases with e)
  const int n_valid = min(E, max(0, (v1 - v0 - (int)threadIdx.x + 255) / 256));
  // start from a valid id, so the argmax stays in the vocabulary even if
  // no value compares greater (NaN logits)
  Top t{-INFINITY, v0, -INFINITY};
  const bool tempered = a.temp != 1.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const float zo = wo * ov[e];
    const float zr = wa * rv[e];
    zv[e] = zo + zr;
    if (tempered) zv[e] = zv[e] / a.temp;
    if (e < n_valid) {
      const int v = v0 + threadIdx.x + e * 256;
      if (z) z[v] = zv[e];
      if (zv[e] > t.m1) {
        t.m2 = t.m1;
        t.m1 = zv[e];
        t.i1 = v;
      } else if (zv[e] > t.m2) {
        t.m2 = zv[e];
      }
    }
  }
  Stat so = stat_of(ov, n_valid), sr = stat_of(rv, n_valid), sz = stat_of(zv, n_valid);
  // wave reduction then LDS across the 4 waves
  for (int off = 32; off > 0; off >>= 1) {
    so = stat_merge(so, stat_shfl(so, off));
    sr = stat_merge(sr, stat_shfl(sr, off));
    sz = stat_merge(sz, stat_shfl(sz, off));
    Top u{__shfl_xor(t.m1, off, 64), __shfl_xor(t.i1, off, 64), __shfl_xor(t.m2, off, 64)};
    t = top_merge(t, u);
  }
  __shared__ Stat sh_st[4][3];
  __shared__ Top sh_top[4];
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sh_st[w][0] = so;
    sh_st[w][1] = sr;
    sh_st[w][2] = sz;
    sh_top[w] = t;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int ww = 1; ww < 4; ++ww) {
      so = stat_merge(so, sh_st[ww][0]);
      sr = stat_merge(sr, sh_st[ww][1]);
      sz = stat_merge(sz, sh_st[ww][2]);
      t = top_merge(t, sh_top[ww]);
    }
    const int R1 = a.R1;
    const Stat st[3] = {so, sr, sz};
    for (int f = 0; f < 3; ++f) {
      float* p = a.part + ((size_t)(f * R1 + row) * a.nchunk + chunk) * 4;
      p[0] = st[f].m;
      p[1] = st[f].s;
      p[2] = st[f].s1;
      p[3] = 0.f;
    }
    float* p = a.part + ((size_t)(3 * R1 + row) * a.nchunk + chunk) * 4;
    p[0] = __int_as_float(t.i1);
    p[1] = t.m1;
    p[2] = t.m2;
    p[3] = 0.f;
  }
}

// One 512-thread workgroup (8 waves) per sequence.  Wave w merges the chunk
// statistics of fused rows w, w+8, ...: lane c takes chunks c and c+64, then
// the wave merges lanes in a fixed butterfly order.  Thread 0 then applies
// the rule.
__global__ __launch_bounds__(512) void k_accept(HeadArgs a) {
  const int b = blockIdx.x, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int kb = a.kb[b], k1 = kb + 1, R1 = a.R1, Kb = kb_prefix(a.kb, b);
  const int zrow0 = b + Kb;  // first fused row of sequence b
  const int* x = a.drafts + (size_t)b * a.k;
  __shared__ int xhat[RV_MAX_DRAFTS + 1];
  __shared__ int xs[RV_MAX_DRAFTS];
  __shared__ float top2[RV_MAX_DRAFTS + 1];
  __shared__ float lse_z[RV_MAX_DRAFTS + 1];
  __shared__ float ent[2][RV_MAX_DRAFTS + 1];
  __shared__ float zx[RV_MAX_DRAFTS];        // fused logit of draft i at row i
  __shared__ float qx[RV_MAX_DRAFTS];        // draft probability of draft i (sampling rule)
  __shared__ float zh[RV_MAX_DRAFTS + 1];    // fused logit of row i's argmax
  // One wave per row (k1 <= 8 with 8 waves): merge the chunk statistics.
  // The same wave also fetches everything the accept decision reads of its
  // row, so the serial tail below touches shared memory only.
  for (int i = w; i < k1; i += 8) {
    const int row = zrow0 + i;
    const int lrow_o = 2 * zrow0 + i, lrow_r = 2 * zrow0 + k1 + i;  // its logit rows
    // draft id and its fused logit / probability, fetched beside the merge
    int xi = 0;
    float zxi = 0.f, qxi = 0.f;
    if (lane == 0 && i < kb) {
      xi = x[i];
      if (xi >= 0 && xi < a.V) {  // out-of-range ids are reported through row_bad
        zxi = fused_at(a, row, lrow_o, lrow_r, xi);
        if (a.rule == RV_RULE_SAMPLING) qxi = a.q[((size_t)b * a.k + i) * a.V + xi];
      }
    }
    Stat st[3] = {{-INFINITY, 0.f, 0.f}, {-INFINITY, 0.f, 0.f}, {-INFINITY, 0.f, 0.f}};
    Top t{-INFINITY, 0x7fffffff, -INFINITY};
    for (int c = lane; c < a.nchunk; c += 64) {
      for (int f = 0; f < 3; ++f) {
        const float* p = a.part + ((size_t)(f * R1 + row) * a.nchunk + c) * 4;
        st[f] = stat_merge(st[f], Stat{p[0], p[1], p[2]});
      }
      const float* pt = a.part + ((size_t)(3 * R1 + row) * a.nchunk + c) * 4;
      t = top_merge(t, Top{pt[1], __float_as_int(pt[0]), pt[2]});
    }
    for (int off = 32; off > 0; off >>= 1) {
      for (int f = 0; f < 3; ++f) st[f] = stat_merge(st[f], stat_shfl(st[f], off));
      Top u{__shfl_xor(t.m1, off, 64), __shfl_xor(t.i1, off, 64), __shfl_xor(t.m2, off, 64)};
      t = top_merge(t, u);
    }
    if (lane == 0) {
      for (int f = 0; f < 3; ++f) a.lse[f * R1 + row] = st[f].m + logf(st[f].s);
      // entropy of the softmax: log S - S1 / S in the centred form
      const float hz = logf(st[2].s) - st[2].s1 / st[2].s;
      const float ho = logf(st[0].s) - st[0].s1 / st[0].s;
      a.entropy[row] = hz;
      a.entropy[R1 + row] = ho;
      ent[0][i] = hz;
      ent[1][i] = ho;
      lse_z[i] = st[2].m + logf(st[2].s);
      t.i1 = min(max(t.i1, 0), a.V - 1);  // every id used as an index below is in range
      xhat[i] = t.i1;
      top2[i] = t.m2;
      zh[i] = fused_at(a, row, lrow_o, lrow_r, t.i1);
      a.argmax[row] = t.i1;
      if (i < kb) {
        xs[i] = xi;
        zx[i] = zxi;
        qx[i] = qxi;
      }
    }
  }
  // any out-of-range id in the sequence's block (or its history) voids it;
  // without a block (logits given by the caller) the draft ids are checked
  int badv = 0;
  if (a.row_bad) {
    const int S = 1 + 2 * kb + a.n_probe + a.P, brow0 = b * (1 + a.n_probe + a.P) + 2 * Kb;
    if (threadIdx.x == 0) badv = a.seq_bad[b];
    for (int j = threadIdx.x; j < S; j += blockDim.x) badv |= a.row_bad[brow0 + j];
  } else {
    for (int j = threadIdx.x; j < kb; j += blockDim.x) badv |= x[j] < 0 || x[j] >= a.V;
  }
  const int bad = __syncthreads_or(badv);
  if (threadIdx.x != 0) return;
  float* mg = a.margins + (size_t)b * (a.k + 2);
  for (int i = 0; i < a.k + 2; ++i) mg[i] = NAN;
  if (bad) {
    a.accept_len[b] = -1;
    a.next_id[b] = -1;
    return;
  }
  int n = kb;
  if (a.rule == RV_RULE_SAMPLING) {
    // reject at the first r_i * q_i(x_i) > p_i(x_i); t is drawn by k_sample
    for (int i = 0; i < kb; ++i) {
      uint64_t c[4] = {(uint64_t)i, (uint64_t)b, 0ull, 0ull};
      philox4x64(c, a.seed, 0ull);
      const float r = uniform23(c[0]);
      const float p = expf(zx[i] - lse_z[i]);
      mg[i] = qx[i] > 0.f ? logf(p) - logf(r * qx[i]) : INFINITY;
      if (r * qx[i] > p) {
        n = i;
        break;
      }
    }
    a.accept_len[b] = n;
    return;
  }
  if (a.rule == RV_RULE_TYPICAL) {
    // log p_i(x_i) > min(log eps, log delta - H_i)  (eps = inf, delta = 0 exact)
    const float log_eps = logf(a.eps), log_delta = logf(a.delta);
    const int src = a.ent_src == RV_ENTROPY_ORIGINAL ? 1 : 0;
    for (int i = 0; i < kb; ++i) {
      const float lp = zx[i] - lse_z[i];
      const float m = lp - fminf(log_eps, log_delta - ent[src][i]);
      mg[i] = m;
      if (!(m > 0.f)) {
        n = i;
        break;
      }
    }
  } else {
    for (int i = 0; i < kb; ++i) {
      if (xhat[i] != xs[i]) {
        n = i;
        break;
      }
    }
    // margins of the tested drafts (inspection only)
    for (int i = 0; i < min(n + 1, kb); ++i) mg[i] = xhat[i] == xs[i] ? zx[i] - top2[i] : zx[i] - zh[i];
  }
  const int t = xhat[n];
  a.accept_len[b] = n;
  a.next_id[b] = t;
  if (a.ids) {  // append x_1..x_n, t to the id history
    const int L = a.L[b];
    int* hist = a.ids + (size_t)b * a.max_len;
    for (int i = 0; i < n; ++i) hist[L + i] = xs[i];
    hist[L + n] = t;
  }
  // bonus-token gap
  mg[a.k + 1] = zh[n] - top2[n];
}

// Sampling rule: one workgroup per (vocabulary chunk, sequence).  Thread
// tid owns the two groups of 4 consecutive ids 4*(tid + 256 u) (u < 2) of
// the chunk, one Philox block each.  Writes the chunk's best perturbed
// score, its lowest id and the runner-up to part plane 3 at the row of
// position n+1.
__global__ __launch_bounds__(256) void k_sample(HeadArgs a) {
  const int chunk = blockIdx.x, b = blockIdx.y;
  const int n = a.accept_len[b];
  if (n < 0) return;
  const int R1 = a.R1, row = b + kb_prefix(a.kb, b) + n;
  const float* z = a.z + (size_t)row * a.V;
  const float lse = a.lse[2 * R1 + row];
  const float* q = n < a.kb[b] ? a.q + ((size_t)b * a.k + n) * a.V : nullptr;
  const int v0 = chunk * a.chunk, v1 = min(a.V, v0 + a.chunk);
  Top t{-INFINITY, v0, -INFINITY};
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int g0 = v0 + 4 * ((int)threadIdx.x + 256 * u);  // a multiple of 4
    if (g0 >= v1) continue;
    uint64_t c[4] = {(uint64_t)(g0 >> 2), (uint64_t)b, 1ull, 0ull};
    philox4x64(c, a.seed, 0ull);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int v = g0 + j;
      if (v >= v1) break;
      const float lz = z[v] - lse;
      float score;
      if (q) {
        const float w = expf(lz) - q[v];
        score = w > 0.f ? logf(w) : -INFINITY;
      } else {
        score = lz;
      }
      const float s = score - logf(-logf(uniform23(c[j])));
      if (s > t.m1) {
        t.m2 = t.m1;
        t.m1 = s;
        t.i1 = v;
      } else if (s > t.m2) {
        t.m2 = s;
      }
    }
  }
  for (int off = 32; off > 0; off >>= 1) {
    Top o{__shfl_xor(t.m1, off, 64), __shfl_xor(t.i1, off, 64), __shfl_xor(t.m2, off, 64)};
    t = top_merge(t, o);
  }
  __shared__ Top sh[4];
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = t;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int ww = 1; ww < 4; ++ww) t = top_merge(t, sh[ww]);
    float* p = a.part + ((size_t)(3 * R1 + row) * a.nchunk + chunk) * 4;
    p[0] = __int_as_float(t.i1);
    p[1] = t.m1;
    p[2] = t.m2;
  }
}

// Sampling rule, one wave per sequence: merges the chunk maxima (lane c
// takes chunks c, c+64, ..., then a fixed butterfly), emits t and appends
// x_1..x_n, t to the id history.
__global__ __launch_bounds__(64) void k_sample_finish(HeadArgs a) {
  const int b = blockIdx.x, lane = threadIdx.x;
  const int n = a.accept_len[b];
  if (n < 0) return;
  const int R1 = a.R1, row = b + kb_prefix(a.kb, b) + n;
  Top t{-INFINITY, 0x7fffffff, -INFINITY};
  for (int c = lane; c < a.nchunk; c += 64) {
    const float* p = a.part + ((size_t)(3 * R1 + row) * a.nchunk + c) * 4;
    t = top_merge(t, Top{p[1], __float_as_int(p[0]), p[2]});
  }
  for (int off = 32; off > 0; off >>= 1) {
    Top o{__shfl_xor(t.m1, off, 64), __shfl_xor(t.i1, off, 64), __shfl_xor(t.m2, off, 64)};
    t = top_merge(t, o);
  }
  if (lane != 0) return;
  const int tok = min(max(t.i1, 0), a.V - 1);
  a.next_id[b] = tok;
  const int* x = a.drafts + (size_t)b * a.k;
  int* hist = a.ids + (size_t)b * a.max_len;
  const int L = a.L[b];
  for (int i = 0; i < n; ++i) hist[L + i] = x[i];
  hist[L + n] = tok;
  a.margins[(size_t)b * (a.k + 2) + a.k + 1] = t.m1 - t.m2;
}

__global__ __launch_bounds__(256) void k_logprob(HeadArgs a) {
  constexpr int E = 8;
  const int chunk = blockIdx.x, fr = blockIdx.y;  // fr = f * R1 + row
  const int R1 = a.R1;
  const int f = fr / R1, row = fr % R1;
  int b, i;
  fused_row_seq(a.kb, a.B, row, b, i);
  const int k1 = a.kb[b] + 1;
  const float* src = f == 2 ? a.z + (size_t)row * a.V
                            : a.logits + ((size_t)2 * (row - i) + (f == 1 ? k1 : 0) + i) * a.V;
  float* dst = a.lp + (size_t)fr * a.V;
  const float l = a.lse[fr];
  const int v0 = chunk * a.chunk, v1 = min(a.V, v0 + a.chunk);
  float x[E];
#pragma unroll
  for (int e = 0; e < E; ++e) x[e] = src[min(v0 + (int)threadIdx.x + e * 256, v1 - 1)];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int v = v0 + threadIdx.x + e * 256;
    if (v < v1) dst[v] = x[e] - l;
  }
}

// dst[i] = exp(src[i]): probabilities from log-probabilities.
__global__ __launch_bounds__(256) void k_exp(const float* __restrict__ src, float* __restrict__ dst, size_t n) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) dst[i] = expf(src[i]);
}

}  // namespace

hipError_t launch_exp(const float* src, float* dst, size_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  k_exp<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(src, dst, n);
  return hipGetLastError();
}

hipError_t launch_head(const HeadArgs& a, hipStream_t st) {
  const int R1 = a.R1;
  k_fuse_stats<<<dim3(a.nchunk, R1), 256, 0, st>>>(a);
  k_accept<<<a.B, 512, 0, st>>>(a);
  if (a.rule == RV_RULE_SAMPLING) {
    k_sample<<<dim3(a.nchunk, a.B), 256, 0, st>>>(a);
    k_sample_finish<<<a.B, 64, 0, st>>>(a);
  }
  if (a.lp) k_logprob<<<dim3(a.nchunk, 3 * R1), 256, 0, st>>>(a);
  return hipGetLastError();
}
