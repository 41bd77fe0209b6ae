// Block assembly, embedding gather, RMSNorm and id-history kernels.
#include "rv_internal.h"

namespace {

// ----------------------------------------------------------- RMSNorm
// y = h * rsqrt(mean(h^2) + eps) * g, stored as a matmul operand; one
// 256-thread workgroup per row.  Pending k-group partials of the previous
// matmul (P, gk) are first added to h in k-group order and h is written back.
template <int DT>
__global__ __launch_bounds__(256) void k_rmsnorm(float* __restrict__ h, int d, const float* __restrict__ gain,
                                                 float eps, void* __restrict__ out, void* __restrict__ out2, int gS,
                                                 int gk, int gshift, const float* __restrict__ P, int pk, int rows) {
  const int r = blockIdx.x;
  int src = r;
  if (gk >= 0) {
    const int per = 2 * (gk + 1), b = r / per, j = r % per;
    src = b * gS + (j <= gk ? j : gshift + j - (gk + 1));
  }
  float* x = h + (size_t)src * d;
  float ss = 0.f;
  for (int i = threadIdx.x * 4; i < d; i += 256 * 4) {
    f32x4_t v = *(const f32x4_t*)(x + i);
    if (P) {
      // batches of 4 independent loads; past the last k-group the load
      // repeats a valid partial and is weighted 0
      for (int g0 = 0; g0 < pk; g0 += 4) {
        f32x4_t pv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) pv[u] = *(const f32x4_t*)(P + ((size_t)min(g0 + u, pk - 1) * rows + src) * d + i);
#pragma unroll
        for (int u = 0; u < 4; ++u) v += g0 + u < pk ? pv[u] : f32x4_t{0.f, 0.f, 0.f, 0.f};
      }
      *(f32x4_t*)(x + i) = v;
    }
    ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
  }
  ss = wave_sum(ss);
  __shared__ float part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = (part[0] + part[1]) + (part[2] + part[3]);
  const float rs = 1.0f / sqrtf(tot / (float)d + eps);
  for (int i = threadIdx.x * 4; i < d; i += 256 * 4) {
    const f32x4_t v = *(const f32x4_t*)(x + i);
    const f32x4_t gg = *(const f32x4_t*)(gain + i);
    f32x4_t o;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = v[j] * rs * gg[j];
    put_operand4<DT>(out, out2, r, i, d, o);
  }
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
template <int DT>
RV_DEV void gather_row(const typename Tr<DT>::T* embed, int tok, int d, float* dst) {
  const typename Tr<DT>::T* e = embed + (size_t)tok * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) dst[i] = Tr<DT>::load(e[i]);
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
  const int L = p.L[b];
  const int* hist = p.ids + (size_t)b * p.max_len;
  int tok;
  if (j == 0) tok = hist[L - 1];
  else if (j <= p.k) tok = p.drafts[b * p.k + j - 1];
  else if (j <= p.k + p.n_probe) tok = p.probe[j - p.k - 1];
  else if (j <= p.k + p.n_probe + p.P) tok = hist[L - p.P + (j - p.k - p.n_probe - 1)];
  else tok = p.drafts[b * p.k + (j - p.k - p.n_probe - p.P - 1)];
  const int row = b * p.S + j;
  const bool bad = tok < 0 || tok >= p.V;
  if (threadIdx.x == 0) {
    p.row_pos[row] = L - 1 + j;
    p.row_seq[row] = b;
    p.row_bad[row] = bad ? 1 : 0;
    if (j == 0) {
      p.seg_b[b] = b;
      p.seg_row0[b] = b * p.S;
      p.seg_n[b] = p.S;
      p.seg_pos0[b] = L - 1;
    }
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
                          void* out2, int gS, int gk, int gshift, const float* P, int pk, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  // partial rows are indexed by source row; the gathering form never reads partials
  if (dtype == RV_BF16)
    k_rmsnorm<RV_BF16><<<rows, 256, 0, st>>>(h, d, gain, eps, out, out2, gS, gk, gshift, P, pk, rows);
  else
    k_rmsnorm<RV_F32><<<rows, 256, 0, st>>>(h, d, gain, eps, out, out2, gS, gk, gshift, P, pk, rows);
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
