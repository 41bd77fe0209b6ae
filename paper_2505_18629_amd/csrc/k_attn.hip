// Block attention against the KV cache.
//
// Every query row at position p of sequence b attends the cached keys
// 0..p of b.  The K/V of the current block were written to the cache by the
// same layer's QKV matmul epilogue (or, after a K-split QKV matmul, by the
// QKV finish kernel), so this causal limit is the whole mask:
// the first draft copy cannot see the probe that follows it (the paper's
// argument for unidirectional attention, Section 3.1), and the probe and
// second copy see everything before them.
//
// Work split: one workgroup per (key split, query group of 128 -- or 192 when
// a kv head has 129-192 queries -- segment x kv head).  The G = Hq/Hkv query
// heads of a kv head share each K/V tile, so a verify block of S rows gives
// G*S queries per kv head (124 for the 8B shape).
// Each split writes unnormalised partial results; a second kernel combines
// splits in a fixed order (deterministic).
#include "rv_internal.h"

namespace {

constexpr int kKB = 64;  // keys per LDS tile

// ----------------------------------------------------------- bf16, MFMA
//
// S^T = K Q^T: A = K unit (16 keys x 32 d), B = Q^T (32 d x 16 queries), so
// lane l holds the scores of keys 4*(l/16)+i for query l%16.
// O^T += V^T P^T: A = V^T unit (16 d x 32 keys), B = P^T taken directly from
// the score registers: hardware k slot j of lane group g is key 4g+j (j < 4)
// of the first 16-key block of a 32-key chunk and key 16+4g+(j-4) of the
// second, the slot order the V cache is stored in.  Q, K, V and P are all
// (hi, lo) bf16 pairs; each product is hi*hi + hi*lo + lo*hi (three MFMAs;
// lo*lo is ~2^-16 of the result and dropped).
//
// The cache keeps K and V in operand order (put_k4 / put_v4), so a 64-key
// tile is four contiguous spans (K hi, K lo, V hi, V lo) that the workgroup
// copies global -> LDS with 16-byte direct loads, double-buffered: tile t+1
// is in flight while tile t is multiplied, and every MFMA operand is one
// conflict-free 16-byte LDS read per lane.  Tiles are 64-aligned and the
// cache holds whole tiles, so copies need no clamping; keys past the valid
// range hold finite values (the cache starts zeroed) and are masked (score
// -inf, so P is exactly 0) or belong to queries whose results are not stored.
template <int HD, int NW, int TPW>
__global__ __launch_bounds__(NW * 64) void k_attn_bf16(AttnArgs a, int n_qg) {
  constexpr int QPW = NW * TPW * 16;          // queries per workgroup
  constexpr int DC = HD / 32;                 // d chunks for QK^T
  constexpr int DT = HD / 16;                 // d tiles for PV
  constexpr int SPAN = kKB * HD;              // elements of one plane of a tile
  constexpr int UNITS = 4 * SPAN / 512;       // 1 KiB units per tile (4 spans)
  constexpr int UPW = (UNITS + NW - 1) / NW;  // units each wave copies (the last round may be partial)
  __shared__ __attribute__((aligned(16))) uint16_t sm0[4][SPAN];
  __shared__ __attribute__((aligned(16))) uint16_t sm1[4][SPAN];

  // Workgroup -> (key split, query group, segment x kv head): the n_qg query
  // groups of one (split, group) read the same K/V tiles, so they get
  // indices 8 apart -- the same XCD (workgroup i runs on XCD i % 8) at about
  // the same time -- and share its L2.
  const int j = blockIdx.x / 8;
  const int unit = (j / n_qg) * 8 + blockIdx.x % 8, qg = j % n_qg;
  if (unit >= a.nsplit * a.nseg * a.n_kv) return;
  const int split = unit % a.nsplit, grp = unit / a.nsplit;
  const int seg = grp / a.n_kv, kvh = grp % a.n_kv;
  const int G = a.n_heads / a.n_kv;
  const int nrows = a.seg_n[seg], row0 = a.seg_row0[seg], pos0 = a.seg_pos0[seg], b = a.seg_b[seg];
  const int Q = G * nrows;
  const int q_begin = qg * QPW;
  if (q_begin >= Q) return;
  const int q_end = min(Q, q_begin + QPW);
  const int kmax = pos0 + (q_end - 1) / G + 1;
  const int kbeg = split * a.ks, kend = min(kmax, kbeg + a.ks);
  const int qpos_min = pos0 + q_begin / G;

  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qd = a.n_heads * HD;
  const size_t kvoff = (size_t)(b * a.n_kv + kvh) * a.kv_len * HD;

  // The units this wave copies: with NW dividing the tile's units, a run of
  // UPW consecutive units (addresses kept per lane); otherwise units w,
  // w + NW, ... (addresses formed per copy).  Unit u is span u / (UNITS/4).
  const uint16_t* src[UNITS % NW == 0 ? UPW : 1];
  int dst[UNITS % NW == 0 ? UPW : 1];
  if constexpr (UNITS % NW == 0) {
#pragma unroll
    for (int i = 0; i < UPW; ++i) {
      const int u = w * UPW + i, sp = u / (UNITS / 4), off = (u % (UNITS / 4)) * 512;
      const void* base = sp == 0 ? a.kc : sp == 1 ? a.kc2 : sp == 2 ? a.vc : a.vc2;
      src[i] = (const uint16_t*)base + kvoff + off + lane * 8;
      dst[i] = sp * SPAN + off;
    }
  }
  auto fetch = [&](uint16_t(&sm)[4][SPAN], int kt0) {
#pragma unroll
    for (int i = 0; i < UPW; ++i) {
      if constexpr (UNITS % NW == 0) {
        __builtin_amdgcn_global_load_lds((const void*)(src[i] + (size_t)kt0 * HD),
                                         (__attribute__((address_space(3))) void*)(&sm[0][0] + dst[i]), 16, 0, 0);
      } else {
        const int u = w + i * NW;
        if (u < UNITS) {
          const int sp = u / (UNITS / 4), off = (u % (UNITS / 4)) * 512;
          const uint16_t* base = (const uint16_t*)(sp == 0 ? a.kc : sp == 1 ? a.kc2 : sp == 2 ? a.vc : a.vc2);
          __builtin_amdgcn_global_load_lds((const void*)(base + kvoff + (size_t)kt0 * HD + off + lane * 8),
                                           (__attribute__((address_space(3))) void*)(&sm[0][0] + sp * SPAN + off),
                                           16, 0, 0);
        }
      }
    }
  };
  if (kbeg < kend) fetch(sm0, kbeg);

  // Queries of this wave: TPW 16-query tiles, hi and lo operand planes.
  uint4 qB[2][TPW][DC];
  int qpos[TPW];
  bool qvalid[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int q = q_begin + (TPW * w + t) * 16 + (lane & 15);
    qvalid[t] = q < q_end;
    const int qc = min(q, q_end - 1);
    qpos[t] = pos0 + qc / G;
    const int row = row0 + qc / G, head = kvh * G + qc % G;
#pragma unroll
    for (int pl = 0; pl < 2; ++pl) {
      const char* qp = (const char*)(pl ? a.q2 : a.q);
#pragma unroll
      for (int c = 0; c < DC; ++c) qB[pl][t][c] = *(const uint4*)(qp + operand_offset(row, head * HD + 32 * c + g * 8, qd, 2));
    }
  }

  float m_run[TPW], l_run[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    m_run[t] = -INFINITY;
    l_run[t] = 0.f;
  }
  f32x4_t O[TPW][DT];
#pragma unroll
  for (int t = 0; t < TPW; ++t)
#pragma unroll
    for (int d = 0; d < DT; ++d) O[t][d] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Waves whose query tiles all lie past q_end (a workgroup of more queries
  // than the segment has) copy their share of each tile and skip the rest.
  const bool active = q_begin + TPW * w * 16 < q_end;

  // One 64-key tile from the LDS buffer sm.
  auto tile = [&](const uint16_t(&sm)[4][SPAN], int kt0) {
    if (!active) return;
    // scores for 64 keys x TPW query tiles
    f32x4_t s[TPW][4];
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) s[t][kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // per 32-dim chunk: the 8 K operands first, then the three products as
    // three passes over the 4 key blocks, so dependent MFMAs are 4 apart
#pragma unroll
    for (int c = 0; c < DC; ++c) {
      bf16x8_t kh[4], kl[4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const int ko = (kt * DC + c) * 512 + lane * 8;
        kh[kt] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(&sm[0][ko]));
        kl[kt] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(&sm[1][ko]));
      }
#pragma unroll
      for (int t = 0; t < TPW; ++t) {
        const bf16x8_t qh = __builtin_bit_cast(bf16x8_t, qB[0][t][c]);
        const bf16x8_t ql = __builtin_bit_cast(bf16x8_t, qB[1][t][c]);
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) s[t][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kh[kt], qh, s[t][kt], 0, 0, 0);
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) s[t][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kh[kt], ql, s[t][kt], 0, 0, 0);
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) s[t][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kl[kt], qh, s[t][kt], 0, 0, 0);
      }
    }

      // online softmax in log2 units: p = 2^(s*scale - m), m the running
      // maximum of the scaled scores (scaling by a positive constant keeps the
      // argmax, so the raw maximum is scaled once).  Interior tiles (every key
      // valid and at or before the earliest query of this workgroup) need no
      // mask; the first tile needs no rescale of the zero accumulators.
      const bool interior = kt0 + kKB <= kend && kt0 + kKB - 1 <= qpos_min;
      const bool first = kt0 == kbeg;
      const float sc = a.scale_log2;
#pragma unroll
      for (int t = 0; t < TPW; ++t) {
        if (!interior) {
#pragma unroll
          for (int kt = 0; kt < 4; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int key = kt0 + 16 * kt + 4 * g + i;
              if (!(key < kend && key <= qpos[t])) s[t][kt][i] = -INFINITY;
            }
        }
        float mloc = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) mloc = fmaxf(mloc, fmaxf(fmaxf(s[t][kt][0], s[t][kt][1]), fmaxf(s[t][kt][2], s[t][kt][3])));
        mloc = rows4_max(mloc);
        const float m_new = fmaxf(m_run[t], mloc * sc);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float rescale = __builtin_amdgcn_exp2f(m_run[t] - m_use);
        float psum = 0.f;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            s[t][kt][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[t][kt][i], sc, -m_use));
            psum += s[t][kt][i];
          }
        psum = rows4_sum(psum);
        l_run[t] = l_run[t] * rescale + psum;
        // rescale is exactly 1 where the maximum did not grow: the wave skips
        // the multiply when that holds for all its lanes
        const bool grew = m_new != m_run[t];
        m_run[t] = m_new;
        if (!first && __any(grew)) {
#pragma unroll
          for (int d = 0; d < DT; ++d) O[t][d] *= rescale;
        }
      }

    // O^T += V^T P^T with P split into hi/lo B operands
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int t = 0; t < TPW; ++t) {
        bf16x8_t phi, plo;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float p = j < 4 ? s[t][2 * c][j] : s[t][2 * c + 1][j - 4];
          const uint16_t hb = f2bf(p);
          const uint16_t lb = f2bf(p - bf2f(hb));
          phi[j] = __builtin_bit_cast(__bf16, hb);
          plo[j] = __builtin_bit_cast(__bf16, lb);
        }
        // the 2*DT V operands first, then the three products as three passes
        // over the d tiles, so dependent MFMAs are DT apart
        bf16x8_t vh[DT], vl[DT];
#pragma unroll
        for (int d = 0; d < DT; ++d) {
          const int vo = (c * DT + d) * 512 + lane * 8;
          vh[d] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(&sm[2][vo]));
          vl[d] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(&sm[3][vo]));
        }
#pragma unroll
        for (int d = 0; d < DT; ++d) O[t][d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vh[d], phi, O[t][d], 0, 0, 0);
#pragma unroll
        for (int d = 0; d < DT; ++d) O[t][d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vh[d], plo, O[t][d], 0, 0, 0);
#pragma unroll
        for (int d = 0; d < DT; ++d) O[t][d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vl[d], phi, O[t][d], 0, 0, 0);
      }
  };

  // Two tiles per iteration so each buffer is named statically.  At the top
  // of each half only the copy of the tile about to be used is in flight;
  // after the barrier every wave has finished the previous tile, so its
  // buffer takes the next copy.
  for (int kt0 = kbeg; kt0 < kend; kt0 += 2 * kKB) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (kt0 + kKB < kend) fetch(sm1, kt0 + kKB);
    tile(sm0, kt0);
    if (kt0 + kKB >= kend) break;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (kt0 + 2 * kKB < kend) fetch(sm0, kt0 + 2 * kKB);
    tile(sm1, kt0 + kKB);
  }

  // Partials: lane holds O^T[d = 16*dt + 4g + i][query lane%16].
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    if (!qvalid[t]) continue;
    const int q = q_begin + (TPW * w + t) * 16 + (lane & 15);
    const size_t e = ((size_t)split * (a.nseg * a.n_kv) + grp) * a.qmax + q;
    float* po = a.part_o + e * HD;
#pragma unroll
    for (int d = 0; d < DT; ++d) *(f32x4_t*)(po + 16 * d + 4 * g) = O[t][d];
    if (g == 0) {
      a.part_ml[2 * e] = m_run[t];
      a.part_ml[2 * e + 1] = l_run[t];
    }
  }
}

// ----------------------------------------------------------- fp32, VALU
// One thread per query; keys read straight from the cache (fp32 models are
// small).  Same partial format as the MFMA kernel.
template <int HD>
__global__ __launch_bounds__(128) void k_attn_f32(AttnArgs a) {
  const int split = blockIdx.x, grp = blockIdx.z;
  const int seg = grp / a.n_kv, kvh = grp % a.n_kv;
  const int G = a.n_heads / a.n_kv;
  const int nrows = a.seg_n[seg], row0 = a.seg_row0[seg], pos0 = a.seg_pos0[seg], b = a.seg_b[seg];
  const int q = blockIdx.y * 128 + threadIdx.x;
  if (q >= G * nrows) return;
  const int qp = pos0 + q / G;
  const int kbeg = split * a.ks, kend = min(qp + 1, kbeg + a.ks);
  const int qrow = row0 + q / G, qcol = (kvh * G + q % G) * HD;
  const float* kb = (const float*)a.kc + (size_t)(b * a.n_kv + kvh) * a.kv_len * HD;
  const float* vb = (const float*)a.vc + (size_t)(b * a.n_kv + kvh) * a.kv_len * HD;
  float qr[HD], o[HD];
#pragma unroll
  for (int d = 0; d < HD; d += 4) {
    const f32x4_t v = *(const f32x4_t*)((const char*)a.q + operand_offset(qrow, qcol + d, a.n_heads * HD, 4));
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      qr[d + i] = v[i];
      o[d + i] = 0.f;
    }
  }
  float m = -INFINITY, l = 0.f;
  for (int key = kbeg; key < kend; ++key) {
    float s = 0.f;
#pragma unroll
    for (int d = 0; d < HD; ++d) s += qr[d] * kb[(size_t)key * HD + d];
    s *= a.scale_log2;
    const float mn = fmaxf(m, s);
    const float r = exp2f(m - mn), p = exp2f(s - mn);
    l = l * r + p;
#pragma unroll
    for (int d = 0; d < HD; ++d) o[d] = o[d] * r + p * vb[(size_t)key * HD + d];
    m = mn;
  }
  const size_t e = ((size_t)split * (a.nseg * a.n_kv) + grp) * a.qmax + q;
#pragma unroll
  for (int d = 0; d < HD; ++d) a.part_o[e * HD + d] = o[d];
  a.part_ml[2 * e] = m;
  a.part_ml[2 * e + 1] = l;
}

// ----------------------------------------------------------- combine
// One wave per query: lane s holds split s's running max and sum (at most 64
// splits), so the merge weights come from two wave reductions; then each lane
// accumulates two output dims over the splits in index order.  The first F
// splits' values are loaded before the reductions, together with the
// statistics (F = 4, 8 or 16, the smallest that covers the query's splits,
// chosen per wave); loads past the last split read a valid duplicate and get
// weight 0, so every load is unconditional; further splits follow in batches
// of 8.
template <int F>
RV_DEV void combine_query(const AttnArgs& a, size_t e0, size_t stride, int ns, int hd, int lane, float& acc0,
                          float& acc1, float& L) {
  const int sl = min(lane, ns - 1);
  const int d0 = min(lane, hd - 1), d1 = min(lane + 64, hd - 1);
  const float ms = a.part_ml[2 * (e0 + sl * stride)];
  const float ls = a.part_ml[2 * (e0 + sl * stride) + 1];
  float w0[F], w1[F];
#pragma unroll
  for (int u = 0; u < F; ++u) {
    const size_t e = e0 + (size_t)min(u, ns - 1) * stride;
    w0[u] = a.part_o[e * hd + d0];
    w1[u] = a.part_o[e * hd + d1];
  }
  const float M = wave_max(lane < ns ? ms : -INFINITY);
  const float f = (lane < ns && ms != -INFINITY) ? exp2f(ms - M) : 0.f;
  L = wave_sum(ls * f);
#pragma unroll
  for (int u = 0; u < F; ++u) {
    const float fu = u < ns ? __shfl(f, u, 64) : 0.f;
    acc0 += w0[u] * fu;
    acc1 += w1[u] * fu;
  }
  for (int s0 = F; s0 < ns; s0 += 8) {
    float v0[8], v1[8], fs[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const size_t e = e0 + (size_t)min(s0 + u, ns - 1) * stride;
      v0[u] = a.part_o[e * hd + d0];
      v1[u] = a.part_o[e * hd + d1];
      fs[u] = __shfl(f, (s0 + u) & 63, 64);
      if (s0 + u >= ns) fs[u] = 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      acc0 += v0[u] * fs[u];
      acc1 += v1[u] * fs[u];
    }
  }
}

template <int DT>
__global__ __launch_bounds__(256) void k_attn_combine(AttnArgs a, int hd) {
  const int lane = threadIdx.x & 63;
  const int grp = blockIdx.y;
  const int seg = grp / a.n_kv, kvh = grp % a.n_kv;
  const int G = a.n_heads / a.n_kv;
  const int q = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int nrows = a.seg_n[seg];
  if (q >= G * nrows) return;
  const int pos_q = a.seg_pos0[seg] + q / G;
  const size_t stride = (size_t)(a.nseg * a.n_kv) * a.qmax;
  const size_t e0 = (size_t)grp * a.qmax + q;
  const int ns = min(a.nsplit, pos_q / a.ks + 1);  // splits that saw keys of this query
  float acc0 = 0.f, acc1 = 0.f, L;
  if (ns <= 4) combine_query<4>(a, e0, stride, ns, hd, lane, acc0, acc1, L);
  else if (ns <= 8) combine_query<8>(a, e0, stride, ns, hd, lane, acc0, acc1, L);
  else combine_query<16>(a, e0, stride, ns, hd, lane, acc0, acc1, L);
  const float inv = 1.0f / L;
  const int row = a.seg_row0[seg] + q / G, head = kvh * G + q % G;
  const int qd = a.n_heads * hd;
  // gather 4 consecutive dims per lane for the operand store
  const float v0 = acc0 * inv, v1 = acc1 * inv;
  const int src = (lane & 15) * 4;  // lanes 0..15 store dims 4l..4l+3 of the first 64, 16..31 of the rest
  f32x4_t x;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float a0 = __shfl(v0, (src + i) & 63, 64);
    const float a1 = __shfl(v1, (src + i) & 63, 64);
    x[i] = lane < 16 ? a0 : a1;
  }
  if (lane < 16 && 4 * lane < hd) put_operand4<DT>(a.out, a.out2, row, head * hd + 4 * lane, qd, x);
  if (lane >= 16 && lane < 32 && 64 + 4 * (lane - 16) < hd)
    put_operand4<DT>(a.out, a.out2, row, head * hd + 64 + 4 * (lane - 16), qd, x);
}

// Row-major copy of cached positions: one thread per (plane, head, position,
// dim) element.
__global__ __launch_bounds__(256) void k_export_kv(const uint16_t* __restrict__ hi, const uint16_t* __restrict__ lo,
                                                   int hd, int n_kv, int kv_len, int pos0, int npos, bool is_v,
                                                   uint16_t* __restrict__ dst) {
  const size_t per_plane = (size_t)n_kv * npos * hd;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= 2 * per_plane) return;
  const int pl = (int)(i / per_plane);
  const size_t r = i % per_plane;
  const int head = (int)(r / ((size_t)npos * hd)), p = (int)(r / hd % npos), d = (int)(r % hd);
  const size_t src = (size_t)head * kv_len * hd + (is_v ? v_elem(pos0 + p, d, hd) : k_elem(pos0 + p, d, hd));
  dst[i] = (pl ? lo : hi)[src];
}

}  // namespace

hipError_t launch_export_kv(const void* src_hi, const void* src_lo, int hd, int n_kv, int kv_len, int pos0,
                            int npos, bool is_v, void* dst, hipStream_t st) {
  const size_t n = (size_t)2 * n_kv * npos * hd;
  if (n == 0) return hipSuccess;
  k_export_kv<<<(unsigned)((n + 255) / 256), 256, 0, st>>>((const uint16_t*)src_hi, (const uint16_t*)src_lo, hd, n_kv,
                                                           kv_len, pos0, npos, is_v, (uint16_t*)dst);
  return hipGetLastError();
}

hipError_t launch_attention(int dtype, const AttnArgs& a, int n_qgroups, int qpw, hipStream_t st) {
  const int groups = a.nseg * a.n_kv;
  if (dtype == RV_BF16) {
    const unsigned units = (unsigned)(a.nsplit * groups);
    const dim3 grid((units + 7) / 8 * 8 * n_qgroups);
    if (qpw != 128 && qpw != 192) return hipErrorInvalidValue;
    const bool w12 = qpw == 192;
    switch (a.hd) {
      case 32:
        if (w12) k_attn_bf16<32, 12, 1><<<grid, 768, 0, st>>>(a, n_qgroups);
        else k_attn_bf16<32, 8, 1><<<grid, 512, 0, st>>>(a, n_qgroups);
        break;
      case 64:
        if (w12) k_attn_bf16<64, 12, 1><<<grid, 768, 0, st>>>(a, n_qgroups);
        else k_attn_bf16<64, 8, 1><<<grid, 512, 0, st>>>(a, n_qgroups);
        break;
      case 128:
        if (w12) k_attn_bf16<128, 12, 1><<<grid, 768, 0, st>>>(a, n_qgroups);
        else k_attn_bf16<128, 8, 1><<<grid, 512, 0, st>>>(a, n_qgroups);
        break;
      default: return hipErrorInvalidValue;
    }
  } else {
    dim3 grid(a.nsplit, (a.qmax + 127) / 128, groups);
    switch (a.hd) {
      case 32: k_attn_f32<32><<<grid, 128, 0, st>>>(a); break;
      case 64: k_attn_f32<64><<<grid, 128, 0, st>>>(a); break;
      case 128: k_attn_f32<128><<<grid, 128, 0, st>>>(a); break;
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

hipError_t launch_attn_combine(int dtype, const AttnArgs& a, hipStream_t st) {
  dim3 grid((a.qmax + 3) / 4, a.nseg * a.n_kv);
  if (dtype == RV_BF16)
    k_attn_combine<RV_BF16><<<grid, 256, 0, st>>>(a, a.hd);
  else
    k_attn_combine<RV_F32><<<grid, 256, 0, st>>>(a, a.hd);
  return hipGetLastError();
}
