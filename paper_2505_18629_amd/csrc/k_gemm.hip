// Weight-streaming matrix kernel: Y[t][p] = sum_k X[t][k] W[p][k] for the
// few-token activations of a verify block (M = batch * block rows) and, with
// more token groups, for prefill chunks.
//
// Layout and schedule
//  - W is packed in 1 KiB tiles of 16 rows x KT k; activations are stored in
//    the matching operand tiles (rv_common.h).  One 16-byte load per lane
//    reads a whole tile, already in MFMA operand order.
//  - A work item is (token group of MTT tiles, row group of NT tiles, k-group
//    of K/GK).  Its 4 waves take interleaved k-steps (wave w: steps
//    kb + w, kb + w + 4, ...) so a workgroup reads one contiguous 4 KiB span
//    of every row tile per step.
//  - Each wave keeps the weight and operand tiles of its next DEPTH k-steps
//    in flight in a register ring.  Loads retire in issue order, so both
//    kinds share the ring depth.
//  - The operand tiles of a k-step are re-read (from L2) by every row group,
//    and those reads compete with the weight stream: with 2 token tiles,
//    8 row tiles per workgroup (ring depth 2) halve them relative to 4.
//  - The 4 per-wave partial tiles are summed in LDS in a fixed order.  With
//    GK > 1 the workgroup writes its fp32 partial tile and the consumer (the
//    next RMSNorm) adds the GK partials in k-group order: deterministic, no
//    atomics.
//  - bf16 models multiply every weight tile by both operand planes (hi, lo).
#include <hip/hip_ext.h>

#include "rv_internal.h"

namespace {

constexpr int kWaves = 4;

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

RV_DEV uint4 load_stream(const uint4* p) {
  const u32x4_t v = __builtin_nontemporal_load((const u32x4_t*)p);
  return uint4{v[0], v[1], v[2], v[3]};
}

RV_DEV float silu(float g) { return g / (1.0f + __expf(-g)); }

template <int DT, int NT, int EPI>
RV_DEV void epilogue(const GemmArgs& a, int tile0, int kg, int tok, int lane, f32x4_t (&v)[NT]) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  const int g = lane >> 4;
  if constexpr (EPI == EPI_STORE || EPI == EPI_RESID) {
    if (tok >= a.M) return;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float* y = a.Y + (size_t)tok * a.ldy + (tile0 + nt) * 16 + 4 * g;
      f32x4_t r = v[nt];
      if constexpr (EPI == EPI_RESID) r += *(const f32x4_t*)y;
      *(f32x4_t*)y = r;
    }
  } else if constexpr (EPI == EPI_PARTIAL) {
    if (tok >= a.M) return;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      *(f32x4_t*)(a.P + ((size_t)kg * a.M + tok) * a.ldy + (tile0 + nt) * 16 + 4 * g) = v[nt];
  } else if constexpr (EPI == EPI_STORE_LOGICAL) {
    if (tok >= a.M) return;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int p = (tile0 + nt) * 16 + 4 * g + i;
        a.Y[(size_t)tok * a.ldy + mat_logical_row(a.md, p)] = v[nt][i];
      }
  } else if constexpr (EPI == EPI_SWIGLU) {
    // physical tile 2t holds gate rows, 2t+1 the matching up rows
    if (tok >= a.M) return;
#pragma unroll
    for (int nt = 0; nt < NT; nt += 2) {
      const int f0 = ((tile0 + nt) >> 1) * 16 + 4 * g;
      f32x4_t out;
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] = silu(v[nt][i]) * v[nt + 1][i];
      put_operand4<DT>(a.act, a.act2, tok, f0, a.N / 2, out);
    }
  } else if constexpr (EPI == EPI_QKV) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      // Rotate-half partner of row r (r < 8) is row r + 8, held by lane ^ 32.
      f32x4_t partner;
#pragma unroll
      for (int i = 0; i < 4; ++i) partner[i] = __shfl_xor(v[nt][i], 32, 64);
      if (tok >= a.M) continue;
      const int p0 = (tile0 + nt) * 16;
      const int pos = a.row_pos[tok];
      if (p0 < a.q_rows + a.k_rows) {
        const bool is_q = p0 < a.q_rows;
        const int rel = is_q ? p0 : p0 - a.q_rows;
        const int head = rel / a.hd, j = (rel % a.hd) >> 4;
        const int half = a.hd >> 1;
        const bool second = lane >= 32;
        const int r0 = 4 * g - (second ? 8 : 0);  // row within the half, 0..7
        const float* cs = a.rope_cos + (size_t)pos * half + 8 * j + r0;
        const float* sn = a.rope_sin + (size_t)pos * half + 8 * j + r0;
        f32x4_t rot;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float c = cs[i], s = sn[i];
          rot[i] = second ? v[nt][i] * c + partner[i] * s : v[nt][i] * c - partner[i] * s;
        }
        const int dim = (second ? half : 0) + 8 * j + r0;
        if (is_q) {
          put_operand4<DT>(a.qbuf, a.qbuf2, tok, head * a.hd + dim, a.n_heads * a.hd, rot);
        } else {
          const int b = a.row_seq[tok];
          put_k4<DT>(a.kc, a.kc2, (size_t)(b * a.n_kv + head) * a.kv_len * a.hd, pos, dim, a.hd, rot);
        }
      } else {
        const int rel = p0 - a.q_rows - a.k_rows + 4 * g;
        const int head = rel / a.hd, dim = rel % a.hd;
        const int b = a.row_seq[tok];
        put_v4<DT>(a.vc, a.vc2, (size_t)(b * a.n_kv + head) * a.kv_len * a.hd, pos, dim, a.hd, v[nt]);
      }
    }
  }
}

template <int DT, int NT, int MTT, int EPI, int kDepth>
__global__ __launch_bounds__(kWaves * 64) void k_gemm(GemmArgs a) {
  using TR = Tr<DT>;
  constexpr int KT = TR::KT;
  constexpr int PL = DT == RV_BF16 ? 2 : 1;
  // weights are read exactly once when a single token group covers M
  constexpr bool kStream = MTT <= 2;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ksteps = a.K / KT;
  const int item = blockIdx.x;
  const int tg = item % a.n_tg, rest = item / a.n_tg;
  const int kg = rest % a.gk, rg = rest / a.gk;
  const int kb = kg * (ksteps / a.gk);
  const int spr = ksteps / (a.gk * kWaves);  // k-steps per wave
  const int tile0 = rg * NT;
  const int tok0 = tg * MTT * 16;

  const uint4* wp = (const uint4*)a.W + (size_t)tile0 * ksteps * 64 + (size_t)(kb + w) * 64 + lane;
  const uint4* xp[PL];
#pragma unroll
  for (int pl = 0; pl < PL; ++pl)
    xp[pl] = (const uint4*)(pl ? a.X2 : a.X) + (size_t)(tok0 >> 4) * ksteps * 64 + (size_t)(kb + w) * 64 + lane;

  f32x4_t acc[NT][MTT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < MTT; ++mt) acc[nt][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  uint4 wq[kDepth][NT], xq[kDepth][PL][MTT];
  // the j-th k-step of this wave is kb + w + 4j
  auto load = [&](int slot, int j) {
    const size_t o = (size_t)j * (kWaves * 64);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const uint4* p = wp + (size_t)nt * ksteps * 64 + o;
      wq[slot][nt] = kStream ? load_stream(p) : *p;
    }
#pragma unroll
    for (int pl = 0; pl < PL; ++pl)
#pragma unroll
      for (int mt = 0; mt < MTT; ++mt) xq[slot][pl][mt] = xp[pl][(size_t)mt * ksteps * 64 + o];
  };
  auto compute = [&](int slot) {
#pragma unroll
    for (int pl = 0; pl < PL; ++pl)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < MTT; ++mt) mma_step<DT>(wq[slot][nt], xq[slot][pl][mt], acc[nt][mt]);
  };
  // Full groups of kDepth steps run branch-free; the last full group only
  // computes; a remainder (spr not a multiple of kDepth) runs unpipelined.
  const int nfull = spr / kDepth;
  int j = 0;
  if (nfull > 0) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) load(d, d);
    for (int gi = 1; gi < nfull; ++gi) {
#pragma unroll
      for (int d = 0; d < kDepth; ++d) {
        compute(d);
        load(d, j + kDepth + d);
      }
      j += kDepth;
    }
#pragma unroll
    for (int d = 0; d < kDepth; ++d) compute(d);
    j += kDepth;
  }
  for (; j < spr; ++j) {
    load(0, j);
    compute(0);
  }

  __shared__ f32x4_t red[kWaves][NT][MTT][64];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < MTT; ++mt) red[w][nt][mt][lane] = acc[nt][mt];
  __syncthreads();
  for (int mt = w; mt < MTT; mt += kWaves) {
    f32x4_t v[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      v[nt] = red[0][nt][mt][lane];
#pragma unroll
      for (int ww = 1; ww < kWaves; ++ww) v[nt] += red[ww][nt][mt][lane];
    }
    epilogue<DT, NT, EPI>(a, tile0, kg, tok0 + mt * 16 + (lane & 15), lane, v);
  }
}

// ------------------------------------------------------------ many tokens
// bf16 only, M > 64 rows (prefill chunks, large batches).  A workgroup owns
// BN = NW * NT * 16 output rows x BM = MT * 16 tokens; its NW = 8 or 12 waves
// (two or three per SIMD, so one wave's LDS and load waits overlap another's MFMAs)
// split the rows (NT tiles each) and share the token tiles: each k-step's
// operand tiles (MT tiles x hi/lo) are staged once per workgroup in
// double-buffered LDS.  Weight tiles go straight to registers (each is used
// by one wave against all MT token tiles).  Both are fetched DEPTH k-steps
// ahead through a register ring.  Workgroups that share rows (the token
// groups of a row group) are given indices that land on one XCD and run
// together, so the weights come from HBM about once.  Every load index is
// clamped, so the pipeline has no branches; rows past M are computed and not
// stored.  (Measured against 4 waves per workgroup, one per SIMD: 8B gate/up
// at 496 tokens 223 -> 153 us, 70B down at 360 tokens 388 -> 262 us.)
// k-steps whose operands are staged per barrier: two for 4 token tiles per
// workgroup (half the barriers; 14B batch 4: 16.77 -> 16.52 ms per pass), one
// for 8 (8B batch 16 measured 18.39 -> 18.57 ms with two)
template <int MT>
constexpr int tiled_kpb() {
  return MT <= 4 ? 2 : 1;
}

template <int NT, int MT, int EPI, int NW, int KPB>
__global__ __launch_bounds__(NW * 64) void k_gemm_tiled(GemmArgs a, int n_rk) {
  constexpr int DEPTH = 4;
  static_assert(DEPTH % (2 * KPB) == 0, "the ring turns over whole pairs of LDS buffers");
  constexpr int XCH = MT * 2 * 64;                     // 16-byte operand chunks per k-step
  constexpr int XU = (XCH + NW * 64 - 1) / (NW * 64);  // per thread (the last round may be partial)
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ksteps = a.K / 32;
  // Item = (row group, k-group) x token group, in an XCD-aware order:
  // workgroup b runs on XCD b % 8, and the n_tg workgroups of one (row group,
  // k-group) share that XCD.  The grid covers n_rk rounded up to a multiple
  // of 8; the workgroups past n_rk have no item.
  const int b = blockIdx.x;
  const int j = b / 8;
  const int rk = (j / a.n_tg) * 8 + b % 8, tg = j % a.n_tg;
  if (rk >= n_rk) return;
  const int rg = rk / a.gk, kg = rk % a.gk;
  const int ks = ksteps / a.gk, kb = kg * ks;  // this k-group's steps
  const int tile0 = (rg * NW + w) * NT;    // this wave's first row tile
  const int last_tt = (a.M - 1) >> 4;          // last valid token tile

  const uint4* wp = (const uint4*)a.W + (size_t)tile0 * ksteps * 64 + (size_t)kb * 64 + lane;
  // operand chunk u of this thread: plane, token tile, lane slot
  const uint4* xsrc[XU];
#pragma unroll
  for (int u = 0; u < XU; ++u) {
    const int c = min((int)threadIdx.x + u * NW * 64, XCH - 1);  // past XCH: a valid chunk, not staged
    const int pl = c / (MT * 64), m = (c / 64) % MT, l16 = c % 64;
    const int tt = min(tg * MT + m, last_tt);
    xsrc[u] = (const uint4*)(pl ? a.X2 : a.X) + ((size_t)tt * ksteps + kb) * 64 + l16;
  }
  __shared__ u32x4 xs[2][KPB][2 * MT * 64];

  f32x4_t acc[NT][MT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[nt][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  u32x4 wq[DEPTH][NT], xq[DEPTH][XU];
  auto load = [&](int slot, int step) {
    step = min(step, ks - 1);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) wq[slot][nt] = *(const u32x4*)(wp + ((size_t)nt * ksteps + step) * 64);
#pragma unroll
    for (int u = 0; u < XU; ++u) xq[slot][u] = *(const u32x4*)(xsrc[u] + (size_t)step * 64);
  };
  auto stage = [&](int slot, int buf, int sub) {
#pragma unroll
    for (int u = 0; u < XU; ++u)
      if (XCH % (NW * 64) == 0 || threadIdx.x + u * NW * 64 < XCH) xs[buf][sub][threadIdx.x + u * NW * 64] = xq[slot][u];
  };
  auto compute = [&](int slot, int buf, int sub) {
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const bf16x8_t xb = __builtin_bit_cast(bf16x8_t, xs[buf][sub][(pl * MT + mt) * 64 + lane]);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wq[slot][nt]), xb,
                                                               acc[nt][mt], 0, 0, 0);
      }
  };

#pragma unroll
  for (int d = 0; d < DEPTH; ++d) load(d, d);
#pragma unroll
  for (int sub = 0; sub < KPB; ++sub) stage(sub, 0, sub);
  __syncthreads();
  // Super-step h of a ring turn (KPB k-steps between barriers): the operands
  // of the next KPB steps go to the other LDS buffer, these KPB steps are
  // computed, and each freed ring slot fetches the step DEPTH ahead.
  for (int s0 = 0; s0 < ks; s0 += DEPTH) {
#pragma unroll
    for (int h = 0; h < DEPTH / KPB; ++h) {
      const int buf = h & 1;
#pragma unroll
      for (int sub = 0; sub < KPB; ++sub) stage(((h + 1) * KPB + sub) % DEPTH, buf ^ 1, sub);
#pragma unroll
      for (int sub = 0; sub < KPB; ++sub) {
        const int d = h * KPB + sub;
        compute(d, buf, sub);
        load(d, s0 + d + DEPTH);
      }
      __syncthreads();
    }
  }

  const int tok_base = tg * MT * 16 + (lane & 15);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    f32x4_t v[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) v[nt] = acc[nt][mt];
    epilogue<RV_BF16, NT, EPI>(a, tile0, kg, tok_base + mt * 16, lane, v);
  }
}

template <int DT, int NT, int MTT, int EPI>
void launch_one(const GemmArgs& a, unsigned items, hipStream_t st) {
  constexpr int kDepth = NT >= 6 ? 2 : 4;
  const dim3 block(kWaves * 64);
  LaunchEvents& ev = g_launch_events;
  if (ev.start) {
    hipExtLaunchKernelGGL(k_gemm<DT, NT, MTT, EPI, kDepth>, dim3(items), block, 0, st, ev.start, ev.stop, 0, a);
    ev = LaunchEvents{};
  } else {
    k_gemm<DT, NT, MTT, EPI, kDepth><<<items, block, 0, st>>>(a);
  }
}

template <int DT, int NT, int EPI>
hipError_t launch_nt(const GemmArgs& a, int mtt, hipStream_t st) {
  const unsigned items = (unsigned)(a.n_tg * a.gk * (a.N / (16 * NT)));
  switch (mtt) {
    case 1: launch_one<DT, NT, 1, EPI>(a, items, st); break;
    case 2: launch_one<DT, NT, 2, EPI>(a, items, st); break;
    case 4:
      if constexpr (NT <= 4) {
        launch_one<DT, NT, 4, EPI>(a, items, st);
        break;
      }
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int DT, int EPI>
hipError_t launch_epi(const GemmArgs& a, int nt, int mtt, hipStream_t st) {
  switch (nt) {
    case 1:
      if constexpr (EPI != EPI_SWIGLU) return launch_nt<DT, 1, EPI>(a, mtt, st);
      break;
    case 2: return launch_nt<DT, 2, EPI>(a, mtt, st);
    case 4: return launch_nt<DT, 4, EPI>(a, mtt, st);
    case 8: return launch_nt<DT, 8, EPI>(a, mtt, st);
    case 3:
    case 6:
      // only K-split launches use 3 or 6 row tiles
      if constexpr (EPI == EPI_PARTIAL) return nt == 3 ? launch_nt<DT, 3, EPI>(a, mtt, st)
                                                       : launch_nt<DT, 6, EPI>(a, mtt, st);
      break;
  }
  return hipErrorInvalidValue;
}

template <int DT>
hipError_t launch_dt(int epi, const GemmArgs& a, int nt, int mtt, hipStream_t st) {
  switch (epi) {
    case EPI_STORE: return launch_epi<DT, EPI_STORE>(a, nt, mtt, st);
    case EPI_RESID: return launch_epi<DT, EPI_RESID>(a, nt, mtt, st);
    case EPI_PARTIAL: return launch_epi<DT, EPI_PARTIAL>(a, nt, mtt, st);
    case EPI_SWIGLU: return launch_epi<DT, EPI_SWIGLU>(a, nt, mtt, st);
    case EPI_QKV: return launch_epi<DT, EPI_QKV>(a, nt, mtt, st);
    case EPI_STORE_LOGICAL: return launch_epi<DT, EPI_STORE_LOGICAL>(a, nt, mtt, st);
  }
  return hipErrorInvalidValue;
}

template <int NT, int MT, int EPI, int NW>
hipError_t launch_tiled_one(const GemmArgs& a, hipStream_t st) {
  const int n_rk = a.N / (16 * NW * NT) * a.gk;
  const unsigned items = (unsigned)((n_rk + 7) / 8 * 8 * a.n_tg);
  const dim3 block(NW * 64);
  LaunchEvents& ev = g_launch_events;
  if (ev.start) {
    hipExtLaunchKernelGGL(k_gemm_tiled<NT, MT, EPI, NW, tiled_kpb<MT>()>, dim3(items), block, 0, st, ev.start, ev.stop, 0,
                          a, n_rk);
    ev = LaunchEvents{};
  } else {
    k_gemm_tiled<NT, MT, EPI, NW, tiled_kpb<MT>()><<<items, block, 0, st>>>(a, n_rk);
  }
  return hipGetLastError();
}

template <int EPI>
hipError_t launch_tiled_epi(const GemmArgs& a, int nw, int nt, int mt, hipStream_t st) {
  if (nw == 8) {
    if (nt == 4 && mt == 8) return launch_tiled_one<4, 8, EPI, 8>(a, st);
    if (nt == 4 && mt == 4) return launch_tiled_one<4, 4, EPI, 8>(a, st);
    if (nt == 2 && mt == 8) return launch_tiled_one<2, 8, EPI, 8>(a, st);
    if (nt == 2 && mt == 4) return launch_tiled_one<2, 4, EPI, 8>(a, st);
    if (nt == 2 && mt == 6) return launch_tiled_one<2, 6, EPI, 8>(a, st);
  } else if (nw == 12) {
    if (nt == 2 && mt == 4) return launch_tiled_one<2, 4, EPI, 12>(a, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm_tiled(int epi, const GemmArgs& a, int nw, int nt, int mt, hipStream_t st) {
  const int ksteps = a.K / 32;
  if (a.gk < 1 || ksteps % a.gk || (ksteps / a.gk) % 4) return hipErrorInvalidValue;
  if (nw < 1 || a.N % (16 * nw * nt)) return hipErrorInvalidValue;
  if (a.gk > 1 && epi != EPI_PARTIAL) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_STORE: return launch_tiled_epi<EPI_STORE>(a, nw, nt, mt, st);
    case EPI_RESID: return launch_tiled_epi<EPI_RESID>(a, nw, nt, mt, st);
    case EPI_PARTIAL: return launch_tiled_epi<EPI_PARTIAL>(a, nw, nt, mt, st);
    case EPI_SWIGLU: return launch_tiled_epi<EPI_SWIGLU>(a, nw, nt, mt, st);
    case EPI_QKV: return launch_tiled_epi<EPI_QKV>(a, nw, nt, mt, st);
    case EPI_STORE_LOGICAL: return launch_tiled_epi<EPI_STORE_LOGICAL>(a, nw, nt, mt, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm(int dtype, int epi, const GemmArgs& a, int nt, int mtt, hipStream_t st) {
  return dtype == RV_BF16 ? launch_dt<RV_BF16>(epi, a, nt, mtt, st) : launch_dt<RV_F32>(epi, a, nt, mtt, st);
}
