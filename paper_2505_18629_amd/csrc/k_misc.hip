// Block assembly, embedding gather, RMSNorm and id-history kernels.
#include <algorithm>

#include "rv_internal.h"

namespace {

// ----------------------------------------------------------- RMSNorm
// y = h * rsqrt(mean(h^2) + eps) * g, stored as a matmul operand.  One
// workgroup of d / (4 NPT) threads per row: every thread owns NPT float4s of
// the row and issues all its loads (the gains, h and the pending k-group
// partials of the previous matmul, added in k-group order) before using any
// of them.  Without a gather the updated h is written back after the
// workgroup's reduction barrier, so the barrier does not wait for that
// store.  With a gather several output rows may read one source row (with no
// probe and no prefix-position tokens, block row k feeds both o_{k+1} and
// r_1), so h is only read: a write-back there would let a workgroup that
// reads after another's store add the partials twice.
// PB: partials loaded per batch, the smallest of 2, 4 and 8 that holds pk
// (larger pk take several batches of 8); loads past pk repeat the last
// partial and are not added.
template <int DT, int NPT, int PB>
__global__ __launch_bounds__(1024) void k_rmsnorm(float* __restrict__ h, int d, const float* __restrict__ gain,
                                                  float eps, void* __restrict__ out, void* __restrict__ out2,
                                                  const int* __restrict__ gather, const float* __restrict__ P,
                                                  int pk, int prows) {
  const int r = blockIdx.x;
  const int src = gather ? gather[r] : r;
  float* x = h + (size_t)src * d;
  f32x4_t v[NPT], gg[NPT];
#pragma unroll
  for (int e = 0; e < NPT; ++e) {
    gg[e] = *(const f32x4_t*)(gain + (threadIdx.x + e * blockDim.x) * 4);
    v[e] = *(const f32x4_t*)(x + (threadIdx.x + e * blockDim.x) * 4);
  }
  if (P) {
    for (int g0 = 0; g0 < pk; g0 += PB) {
      f32x4_t pv[NPT][PB];
#pragma unroll
      for (int e = 0; e < NPT; ++e)
#pragma unroll
        for (int u = 0; u < PB; ++u)
          pv[e][u] = *(const f32x4_t*)(P + ((size_t)min(g0 + u, pk - 1) * prows + src) * d +
                                       (threadIdx.x + e * blockDim.x) * 4);
#pragma unroll
      for (int e = 0; e < NPT; ++e)
#pragma unroll
        for (int u = 0; u < PB; ++u) v[e] += g0 + u < pk ? pv[e][u] : f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int e = 0; e < NPT; ++e) ss += v[e][0] * v[e][0] + v[e][1] * v[e][1] + v[e][2] * v[e][2] + v[e][3] * v[e][3];
  ss = wave_sum(ss);
  __shared__ float part[16];
  const int nw = blockDim.x >> 6;
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
  for (int w = 0; w < nw; ++w) tot += part[w];
  const float rs = 1.0f / sqrtf(tot / (float)d + eps);
  if (P && !gather) {
#pragma unroll
    for (int e = 0; e < NPT; ++e) *(f32x4_t*)(x + (threadIdx.x + e * blockDim.x) * 4) = v[e];
  }
#pragma unroll
  for (int e = 0; e < NPT; ++e) {
    const int i = (threadIdx.x + e * blockDim.x) * 4;
    f32x4_t o;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = v[e][j] * rs * gg[e][j];
    put_operand4<DT>(out, out2, r, i, d, o);
  }
}

// One finish unit: token tok, 16-row tile `tile` of the packed QKV matrix,
// rows r0..r0+3 (r0 in {0, 4}) and their rotate-half partners r0+8..r0+11.
// Sums the k-group partials in order, applies rotary to q and k rows, and
// writes the q operand or the K/V cache rows.  The first PB k-groups' loads
// are issued before the token's position is read (they do not depend on
// it), so the rotary table loads are the only dependent round trip.
template <int DT, int PB>
RV_DEV void qkv_finish_unit(const QkvFinish& a, int tok, int tile, int r0) {
  const int p0 = tile * 16;
  auto part = [&](int g) { return a.P + ((size_t)g * a.M + tok) * a.N + p0; };
  f32x4_t l1[PB], l2[PB];
#pragma unroll
  for (int v = 0; v < PB; ++v) {
    const float* row = part(min(v, a.gk - 1));
    l1[v] = *(const f32x4_t*)(row + r0);
    l2[v] = *(const f32x4_t*)(row + 8 + r0);
  }
  const int pos = a.row_pos[tok], b = a.row_seq[tok];
  f32x4_t x1 = {0.f, 0.f, 0.f, 0.f}, x2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int v = 0; v < PB; ++v) {
    if (v < a.gk) {
      x1 += l1[v];
      x2 += l2[v];
    }
  }
  for (int g0 = PB; g0 < a.gk; g0 += 8) {  // more than PB (= 8) k-groups
    f32x4_t m1[8], m2[8];
#pragma unroll
    for (int v = 0; v < 8; ++v) {
      const float* row = part(min(g0 + v, a.gk - 1));
      m1[v] = *(const f32x4_t*)(row + r0);
      m2[v] = *(const f32x4_t*)(row + 8 + r0);
    }
#pragma unroll
    for (int v = 0; v < 8; ++v) {
      if (g0 + v < a.gk) {
        x1 += m1[v];
        x2 += m2[v];
      }
    }
  }
  const int half = a.hd / 2;
  if (p0 < a.q_rows + a.k_rows) {
    const bool is_q = p0 < a.q_rows;
    const int rel = is_q ? p0 : p0 - a.q_rows;
    const int head = rel / a.hd, j = (rel % a.hd) >> 4;
    const f32x4_t cs = *(const f32x4_t*)(a.rope_cos + (size_t)pos * half + 8 * j + r0);
    const f32x4_t sn = *(const f32x4_t*)(a.rope_sin + (size_t)pos * half + 8 * j + r0);
    f32x4_t o1, o2;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o1[i] = x1[i] * cs[i] - x2[i] * sn[i];
      o2[i] = x2[i] * cs[i] + x1[i] * sn[i];
    }
    const int d1 = 8 * j + r0, d2 = half + 8 * j + r0;
    if (is_q) {
      put_operand4<DT>(a.qbuf, a.qbuf2, tok, head * a.hd + d1, a.n_heads * a.hd, o1);
      put_operand4<DT>(a.qbuf, a.qbuf2, tok, head * a.hd + d2, a.n_heads * a.hd, o2);
    } else {
      const size_t kb = (size_t)(b * a.n_kv + head) * a.kv_len * a.hd;
      put_k4<DT>(a.kc, a.kc2, kb, pos, d1, a.hd, o1);
      put_k4<DT>(a.kc, a.kc2, kb, pos, d2, a.hd, o2);
    }
  } else {
    const int rel = p0 - a.q_rows - a.k_rows;
    const int head = rel / a.hd, dim = rel % a.hd;
    const size_t vb = (size_t)(b * a.n_kv + head) * a.kv_len * a.hd;
    put_v4<DT>(a.vc, a.vc2, vb, pos, dim + r0, a.hd, x1);
    put_v4<DT>(a.vc, a.vc2, vb, pos, dim + 8 + r0, a.hd, x2);
  }
}

// Completes a K-split QKV projection: sums the k-group partials (physical
// row order of the packed QKV matrix) in order, applies rotate-half rotary to
// q and k, and writes the q operand and the K/V cache rows.  Workgroups of
// 256 threads, gridDim.y of them per token; a thread handles rows r0..r0+3
// of a 16-row tile and their rotary partners r0+8..r0+11 (r0 in {0, 4}).
template <int DT, int PB>
__global__ __launch_bounds__(256) void k_qkv_finish(QkvFinish a) {
  const int tok = blockIdx.x;
  const int units = a.N / 8;
  for (int u = blockIdx.y * blockDim.x + threadIdx.x; u < units; u += gridDim.y * blockDim.x)
    qkv_finish_unit<DT, PB>(a, tok, u >> 1, (u & 1) * 4);
}

// Row-major [rows][K] <-> operand tiles, one element per thread.
template <typename T>
__global__ void k_retile(const T* __restrict__ src, T* __restrict__ dst, int rows, int K, bool to_tiles) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (size_t)rows * K) return;
  const int t = (int)(i / K), k = (int)(i % K);
  const size_t o = operand_offset(t, k, K, sizeof(T)) / sizeof(T);
  if (to_tiles) dst[o] = src[i];
  else dst[i] = src[o];
}

// ----------------------------------------------------------- embedding gather
// d is a multiple of 128: each thread moves 8 (bf16) or 4 (fp32) elements
// per 16-byte load.
template <int DT>
RV_DEV void gather_row(const typename Tr<DT>::T* embed, int tok, int d, float* dst) {
  using T = typename Tr<DT>::T;
  constexpr int V = 16 / sizeof(T);
  const T* e = embed + (size_t)tok * d;
  for (int i = threadIdx.x * V; i < d; i += blockDim.x * V) {
    const u32x4 raw = *(const u32x4*)(e + i);
    if constexpr (DT == RV_BF16) {
      f32x4_t lo, hi;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        lo[j] = __uint_as_float(raw[j] << 16);
        hi[j] = __uint_as_float(raw[j] & 0xffff0000u);
      }
      // element 2j is the low half of word j
      *(f32x4_t*)(dst + i) = f32x4_t{lo[0], hi[0], lo[1], hi[1]};
      *(f32x4_t*)(dst + i + 4) = f32x4_t{lo[2], hi[2], lo[3], hi[3]};
    } else {
      *(f32x4_t*)(dst + i) = __builtin_bit_cast(f32x4_t, raw);
    }
  }
}

// Verify block, one workgroup per (row j, sequence b):
//   j = 0            c = ids[L-1]
//   j = 1..k         x_j
//   then n_probe     probe ids
//   then P           ids[L-P .. L-1]
//   then k           x_1..x_k again                         (Eq. 1)
// at positions L-1+j.
template <int DT>
__global__ __launch_bounds__(256) void k_plan_verify(PlanVerify p) {
  const int j = blockIdx.x, b = blockIdx.y;
  const int k = p.kb[b], S = 1 + 2 * k + p.n_probe + p.P;
  if (j >= S) return;
  const int Kb = kb_prefix(p.kb, b);
  const int row0 = b * (1 + p.n_probe + p.P) + 2 * Kb;  // first block row of sequence b
  const int L = p.L[b];
  const int* hist = p.ids + (size_t)b * p.max_len;
  const int* x = p.drafts + (size_t)b * p.k;
  int tok;
  if (j == 0) tok = hist[L - 1];
  else if (j <= k) tok = x[j - 1];
  else if (j <= k + p.n_probe) tok = p.probe[j - k - 1];
  else if (j <= k + p.n_probe + p.P) tok = hist[L - p.P + (j - k - p.n_probe - 1)];
  else tok = x[j - k - p.n_probe - p.P - 1];
  const int row = row0 + j;
  const bool bad = tok < 0 || tok >= p.V;
  if (threadIdx.x == 0) {
    p.row_pos[row] = L - 1 + j;
    p.row_seq[row] = b;
    p.row_bad[row] = bad ? 1 : 0;
    if (j == 0) {
      p.seg_b[b] = b;
      p.seg_row0[b] = row0;
      p.seg_n[b] = S;
      p.seg_pos0[b] = L - 1;
    }
    // LM-head rows of sequence b: o_1..o_{k+1} = block rows 0..k, then
    // r_1..r_{k+1} = rows shift..shift+k (shift = k + n_probe + P)
    const int lrow0 = 2 * (b + Kb), shift = k + p.n_probe + p.P;
    if (j <= k) p.lm_src[lrow0 + j] = row;
    if (j >= shift && j <= shift + k) p.lm_src[lrow0 + k + 1 + (j - shift)] = row;
  }
  gather_row<DT>((const typename Tr<DT>::T*)p.embed, bad ? 0 : tok, p.d, p.h + (size_t)row * p.d);
}

// Prefill chunk: one workgroup per row.
template <int DT>
__global__ __launch_bounds__(256) void k_plan_prefill(PlanPrefill p) {
  const int row = blockIdx.x;
  int s = 0;
  while (s + 1 < p.nseg && p.srow0[s + 1] <= row) ++s;
  const int b = p.sb[s], pos = p.spos0[s] + (row - p.srow0[s]);
  int tok = p.prefix[(size_t)b * p.ld + pos];
  if (tok < 0 || tok >= p.V) tok = 0;  // reported through the sequence flag
  if (threadIdx.x == 0) {
    p.row_pos[row] = pos;
    p.row_seq[row] = b;
    if (row == p.srow0[s]) {
      p.seg_b[s] = b;
      p.seg_row0[s] = p.srow0[s];
      p.seg_n[s] = p.sn[s];
      p.seg_pos0[s] = p.spos0[s];
    }
  }
  gather_row<DT>((const typename Tr<DT>::T*)p.embed, tok, p.d, p.h + (size_t)row * p.d);
}

// Copies the committed ids into the history and sets the per-sequence flag
// of out-of-range ids; one workgroup per sequence.
__global__ __launch_bounds__(256) void k_store_ids(StoreIds s) {
  const int b = blockIdx.x, L = s.L[b];
  int bad = 0;
  for (int i = threadIdx.x; i < L; i += 256) {
    const int t = s.prefix[(size_t)b * s.ld + i];
    bad |= (t < 0 || t >= s.V);
    s.ids[(size_t)b * s.max_len + i] = t;
  }
  bad = __syncthreads_or(bad);
  if (threadIdx.x == 0) s.seq_bad[b] = bad;
}

}  // namespace

hipError_t launch_rmsnorm(int dtype, float* h, int rows, int d, const float* gain, float eps, void* out,
                          void* out2, const int* gather, const float* P, int pk, int prows, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  // d is a multiple of 128: one float4 per thread up to d = 4096, else two
  const int npt = d <= 4096 ? 1 : 2;
  const int threads = d / (4 * npt);
  if (threads > 1024 || threads % 64) return hipErrorInvalidValue;
  const int pb = pk <= 2 ? 2 : pk <= 4 ? 4 : 8;
#define RV_NORM(DT_, N_, PB_) \
  k_rmsnorm<DT_, N_, PB_><<<rows, threads, 0, st>>>(h, d, gain, eps, out, out2, gather, P, pk, prows)
#define RV_NORM_PB(DT_, N_)       \
  if (pb == 2) RV_NORM(DT_, N_, 2); \
  else if (pb == 4) RV_NORM(DT_, N_, 4); \
  else RV_NORM(DT_, N_, 8)
  if (dtype == RV_BF16) {
    if (npt == 1) { RV_NORM_PB(RV_BF16, 1); } else { RV_NORM_PB(RV_BF16, 2); }
  } else {
    if (npt == 1) { RV_NORM_PB(RV_F32, 1); } else { RV_NORM_PB(RV_F32, 2); }
  }
#undef RV_NORM_PB
#undef RV_NORM
  return hipGetLastError();
}

hipError_t launch_qkv_finish(int dtype, const QkvFinish& a, hipStream_t st) {
  // workgroups of 256 threads, one unit each, spread over as many
  // workgroups per token as the units need (8B: 768 units, 3 per token)
  const int units = a.N / 8;
  const dim3 grid(a.M, (units + 255) / 256);
  const int pb = a.gk <= 2 ? 2 : a.gk <= 4 ? 4 : 8;
#define RV_FIN(DT_, PB_) k_qkv_finish<DT_, PB_><<<grid, 256, 0, st>>>(a)
  if (dtype == RV_BF16) {
    if (pb == 2) RV_FIN(RV_BF16, 2); else if (pb == 4) RV_FIN(RV_BF16, 4); else RV_FIN(RV_BF16, 8);
  } else {
    if (pb == 2) RV_FIN(RV_F32, 2); else if (pb == 4) RV_FIN(RV_F32, 4); else RV_FIN(RV_F32, 8);
  }
#undef RV_FIN
  return hipGetLastError();
}

hipError_t launch_retile(int dtype, const void* src, void* dst, int rows, int K, bool to_tiles, hipStream_t st) {
  const size_t n = (size_t)rows * K;
  const dim3 grid((unsigned)((n + 255) / 256));
  if (dtype == RV_BF16)
    k_retile<uint16_t><<<grid, 256, 0, st>>>((const uint16_t*)src, (uint16_t*)dst, rows, K, to_tiles);
  else
    k_retile<float><<<grid, 256, 0, st>>>((const float*)src, (float*)dst, rows, K, to_tiles);
  return hipGetLastError();
}

hipError_t launch_plan_verify(int dtype, const PlanVerify& p, hipStream_t st) {
  dim3 grid(p.S, p.B);
  if (dtype == RV_BF16)
    k_plan_verify<RV_BF16><<<grid, 256, 0, st>>>(p);
  else
    k_plan_verify<RV_F32><<<grid, 256, 0, st>>>(p);
  return hipGetLastError();
}

hipError_t launch_plan_prefill(int dtype, const PlanPrefill& p, hipStream_t st) {
  if (dtype == RV_BF16)
    k_plan_prefill<RV_BF16><<<p.rows, 256, 0, st>>>(p);
  else
    k_plan_prefill<RV_F32><<<p.rows, 256, 0, st>>>(p);
  return hipGetLastError();
}

hipError_t launch_store_ids(const StoreIds& s, hipStream_t st) {
  k_store_ids<<<s.B, 256, 0, st>>>(s);
  return hipGetLastError();
}
