// Fusion, log-softmax and the accept decision of one verify pass.
//
//  1. k_fuse_stats   z_i = (1 - alpha) o_i + alpha r_i (Eq. 2, fp32, no FMA
//                    contraction, so alpha = 0 and alpha = 1 give o and r
//                    exactly) and, per vocabulary chunk, the running max and
//                    sum of exp for o, r and z plus z's top-2 and argmax.
//  2. k_accept       per sequence: merges the chunks in index order, takes
//                    x_hat_i = argmax z_i (lowest id on ties), accepts the
//                    leading drafts equal to x_hat (Algorithm 2 at
//                    temperature 0), emits t = x_hat_{n+1}, appends
//                    x_1..x_n, t to the id history.
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

RV_DEV void lse_merge(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;
  s = s * __expf(m - mn) + s2 * __expf(m2 - mn);
  m = mn;
}

RV_DEV void lse_add(float& m, float& s, float x) {
  if (x > m) {
    s = s * __expf(m - x) + 1.0f;
    m = x;
  } else {
    s += __expf(x - m);
  }
}

// One workgroup per (vocabulary chunk of 2048, fused row); each thread owns 8
// entries and loads them all before computing.
__global__ __launch_bounds__(256) void k_fuse_stats(HeadArgs a) {
  constexpr int E = 8;
  const int chunk = blockIdx.x, row = blockIdx.y;  // row = b*(k+1) + i
  const int k1 = a.k + 1, b = row / k1, i = row % k1;
  const float* o = a.logits + ((size_t)b * 2 * k1 + i) * a.V;
  const float* r = a.logits + ((size_t)b * 2 * k1 + k1 + i) * a.V;
  float* z = a.z + (size_t)row * a.V;
  const float wa = a.alpha, wo = 1.0f - a.alpha;
  const int v0 = chunk * a.chunk, v1 = min(a.V, v0 + a.chunk);
  float ov[E], rv[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int v = min(v0 + threadIdx.x + e * 256, v1 - 1);
    ov[e] = o[v];
    rv[e] = r[v];
  }
  float mo = -INFINITY, so = 0.f, mr = -INFINITY, sr = 0.f, mz = -INFINITY, sz = 0.f;
  // start from a valid id, so the argmax stays in the vocabulary even if
  // no value compares greater (NaN logits)
  Top t{-INFINITY, v0, -INFINITY};
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int v = v0 + threadIdx.x + e * 256;
    if (v >= v1) continue;
    const float zo = wo * ov[e];
    const float zr = wa * rv[e];
    const float zv = zo + zr;
    z[v] = zv;
    lse_add(mo, so, ov[e]);
    lse_add(mr, sr, rv[e]);
    lse_add(mz, sz, zv);
    if (zv > t.m1) {
      t.m2 = t.m1;
      t.m1 = zv;
      t.i1 = v;
    } else if (zv > t.m2) {
      t.m2 = zv;
    }
  }
  // wave reduction then LDS across the 4 waves
  for (int off = 32; off > 0; off >>= 1) {
    lse_merge(mo, so, __shfl_xor(mo, off, 64), __shfl_xor(so, off, 64));
    lse_merge(mr, sr, __shfl_xor(mr, off, 64), __shfl_xor(sr, off, 64));
    lse_merge(mz, sz, __shfl_xor(mz, off, 64), __shfl_xor(sz, off, 64));
    Top u{__shfl_xor(t.m1, off, 64), __shfl_xor(t.i1, off, 64), __shfl_xor(t.m2, off, 64)};
    t = top_merge(t, u);
  }
  __shared__ float sh[4][9];
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sh[w][0] = mo; sh[w][1] = so; sh[w][2] = mr; sh[w][3] = sr; sh[w][4] = mz; sh[w][5] = sz;
    sh[w][6] = t.m1; sh[w][7] = __int_as_float(t.i1); sh[w][8] = t.m2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int ww = 1; ww < 4; ++ww) {
      lse_merge(mo, so, sh[ww][0], sh[ww][1]);
      lse_merge(mr, sr, sh[ww][2], sh[ww][3]);
      lse_merge(mz, sz, sh[ww][4], sh[ww][5]);
      t = top_merge(t, Top{sh[ww][6], __float_as_int(sh[ww][7]), sh[ww][8]});
    }
    const int R1 = a.B * k1;
    float* p0 = a.part + ((size_t)(0 * R1 + row) * a.nchunk + chunk) * 4;
    float* p1 = a.part + ((size_t)(1 * R1 + row) * a.nchunk + chunk) * 4;
    float* p2 = a.part + ((size_t)(2 * R1 + row) * a.nchunk + chunk) * 4;
    p0[0] = mo; p0[1] = so;
    p1[0] = mr; p1[1] = sr;
    p2[0] = mz; p2[1] = sz; p2[2] = __int_as_float(t.i1); p2[3] = t.m1;
    // second value is kept in the o slot's spare fields
    p0[2] = t.m2;
  }
}

// One 256-thread workgroup per sequence.  Wave w merges the chunk statistics
// of fused rows w, w+4, ...: lane c takes chunks c and c+64, then the wave
// merges lanes in a fixed butterfly order.  Thread 0 then applies the rule.
__global__ __launch_bounds__(256) void k_accept(HeadArgs a) {
  const int b = blockIdx.x, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int k1 = a.k + 1, R1 = a.B * k1;
  __shared__ int xhat[RV_MAX_DRAFTS + 1];
  __shared__ float top2[RV_MAX_DRAFTS + 1];
  for (int i = w; i < k1; i += 4) {
    const int row = b * k1 + i;
    float m[3] = {-INFINITY, -INFINITY, -INFINITY}, s[3] = {0.f, 0.f, 0.f};
    Top t{-INFINITY, 0x7fffffff, -INFINITY};
    for (int c = lane; c < a.nchunk; c += 64) {
      for (int f = 0; f < 3; ++f) {
        const float* p = a.part + ((size_t)(f * R1 + row) * a.nchunk + c) * 4;
        lse_merge(m[f], s[f], p[0], p[1]);
      }
      const float* pz = a.part + ((size_t)(2 * R1 + row) * a.nchunk + c) * 4;
      const float* po = a.part + ((size_t)(0 * R1 + row) * a.nchunk + c) * 4;
      t = top_merge(t, Top{pz[3], __float_as_int(pz[2]), po[2]});
    }
    for (int off = 32; off > 0; off >>= 1) {
      for (int f = 0; f < 3; ++f) lse_merge(m[f], s[f], __shfl_xor(m[f], off, 64), __shfl_xor(s[f], off, 64));
      Top u{__shfl_xor(t.m1, off, 64), __shfl_xor(t.i1, off, 64), __shfl_xor(t.m2, off, 64)};
      t = top_merge(t, u);
    }
    if (lane == 0) {
      for (int f = 0; f < 3; ++f) a.lse[f * R1 + row] = m[f] + logf(s[f]);
      t.i1 = min(max(t.i1, 0), a.V - 1);  // every id used as an index below is in range
      xhat[i] = t.i1;
      top2[i] = t.m2;
      a.argmax[row] = t.i1;
    }
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  int bad = a.seq_bad[b];
  for (int j = 0; j < a.S; ++j) bad |= a.row_bad[b * a.S + j];
  if (bad) {
    a.accept_len[b] = -1;
    a.next_id[b] = -1;
    return;
  }
  const int* x = a.drafts + (size_t)b * a.k;
  int n = a.k;
  for (int i = 0; i < a.k; ++i) {
    if (xhat[i] != x[i]) {
      n = i;
      break;
    }
  }
  const int t = xhat[n];
  a.accept_len[b] = n;
  a.next_id[b] = t;
  const int L = a.L[b];
  int* hist = a.ids + (size_t)b * a.max_len;
  for (int i = 0; i < n; ++i) hist[L + i] = x[i];
  hist[L + n] = t;
  // margins of the tested drafts and the bonus-token gap (inspection only)
  float* mg = a.margins + (size_t)b * (a.k + 2);
  for (int i = 0; i < a.k + 2; ++i) mg[i] = NAN;
  for (int i = 0; i < min(n + 1, a.k); ++i) {
    const float* zi = a.z + ((size_t)b * k1 + i) * a.V;
    const float zx = zi[x[i]];
    const float top = zi[xhat[i]];
    mg[i] = xhat[i] == x[i] ? zx - top2[i] : zx - top;
  }
  mg[a.k + 1] = a.z[((size_t)b * k1 + n) * a.V + t] - top2[n];
}

__global__ __launch_bounds__(256) void k_logprob(HeadArgs a) {
  constexpr int E = 8;
  const int chunk = blockIdx.x, fr = blockIdx.y;  // fr = f * R1 + row
  const int k1 = a.k + 1, R1 = a.B * k1;
  const int f = fr / R1, row = fr % R1, b = row / k1, i = row % k1;
  const float* src = f == 2 ? a.z + (size_t)row * a.V
                            : a.logits + ((size_t)b * 2 * k1 + (f == 1 ? k1 : 0) + i) * a.V;
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

}  // namespace

hipError_t launch_head(const HeadArgs& a, hipStream_t st) {
  const int R1 = a.B * (a.k + 1);
  k_fuse_stats<<<dim3(a.nchunk, R1), 256, 0, st>>>(a);
  k_accept<<<a.B, 256, 0, st>>>(a);
  k_logprob<<<dim3(a.nchunk, 3 * R1), 256, 0, st>>>(a);
  return hipGetLastError();
}
