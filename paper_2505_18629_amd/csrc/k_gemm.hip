// Weight-streaming matrix kernel: Y[t][p] = sum_k X[t][k] W[p][k] for the
// few-row activations of a verify block (M = batch * block rows).
//
// Layout and schedule
//  - W is packed in 1 KiB tiles of 16 rows x KT k (see rv_common.h): one
//    16-byte load per lane reads a whole tile, fully coalesced, already in
//    MFMA operand order.  Each weight byte is read from HBM once per launch.
//  - A workgroup owns NT consecutive 16-row tiles and MTT 16-token tiles and
//    splits K over its 8 waves; the per-wave partial tiles are summed in LDS
//    in a fixed order (deterministic, no atomics).
//  - grid.x walks token groups fastest, so launches with more tokens than
//    one workgroup covers re-read each weight tile from L2, not HBM.
//  - The epilogue runs on the reduced tile in MFMA output layout: lane l
//    holds rows 4*(l/16)+i (i = 0..3) of token l%16.
#include "rv_internal.h"

namespace {

constexpr int kWaves = 8;

RV_DEV float silu(float g) { return g / (1.0f + __expf(-g)); }

template <int DT, int NT, int EPI>
RV_DEV void epilogue(const GemmArgs& a, int tile0, int tok, int lane, f32x4_t (&v)[NT]) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  const int g = lane >> 4;
  if constexpr (EPI == EPI_STORE || EPI == EPI_RESID) {
    if (tok >= a.M) return;
    float* y = a.Y + (size_t)tok * a.ldy + tile0 * 16 + 4 * g;
    f32x4_t r = v[0];
    if constexpr (EPI == EPI_RESID) r += *(const f32x4_t*)y;
    *(f32x4_t*)y = r;
  } else if constexpr (EPI == EPI_STORE_LOGICAL) {
    if (tok >= a.M) return;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int p = tile0 * 16 + 4 * g + i;
      a.Y[(size_t)tok * a.ldy + mat_logical_row(a.md, p)] = v[0][i];
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    if (tok >= a.M) return;
    const int f0 = (tile0 >> 1) * 16 + 4 * g;
    f32x4_t out;
#pragma unroll
    for (int i = 0; i < 4; ++i) out[i] = silu(v[0][i]) * v[1][i];
    put_operand4<DT>(a.act, a.act2, (size_t)tok * a.ld_act + f0, out);
  } else if constexpr (EPI == EPI_QKV) {
    // Rotate-half partner of row r (r < 8) is row r + 8, held by lane ^ 32.
    f32x4_t partner;
#pragma unroll
    for (int i = 0; i < 4; ++i) partner[i] = __shfl_xor(v[0][i], 32, 64);
    if (tok >= a.M) return;
    const int p0 = tile0 * 16;
    const int pos = a.row_pos[tok];
    T out[4];
    if (p0 < a.q_rows + a.k_rows) {
      const bool is_q = p0 < a.q_rows;
      const int rel = is_q ? p0 : p0 - a.q_rows;
      const int head = rel / a.hd, j = (rel % a.hd) >> 4;
      const int half = a.hd >> 1;
      const bool second = lane >= 32;
      const int r0 = 4 * g - (second ? 8 : 0);      // row within the half, 0..7
      const float* cs = a.rope_cos + (size_t)pos * half + 8 * j + r0;
      const float* sn = a.rope_sin + (size_t)pos * half + 8 * j + r0;
      f32x4_t rot;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float c = cs[i], s = sn[i];
        rot[i] = second ? v[0][i] * c + partner[i] * s : v[0][i] * c - partner[i] * s;
      }
      const int dim = (second ? half : 0) + 8 * j + r0;
      if (is_q) {
        put_operand4<DT>(a.qbuf, a.qbuf2, (size_t)tok * (a.n_heads * a.hd) + head * a.hd + dim, rot);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) out[i] = TR::store(rot[i]);
        const int b = a.row_seq[tok];
        memcpy((T*)a.kc + ((size_t)(b * a.n_kv + head) * a.max_len + pos) * a.hd + dim, out, sizeof(out));
      }
    } else {
      const int rel = p0 - a.q_rows - a.k_rows + 4 * g;
      const int head = rel / a.hd, dim = rel % a.hd;
      const int b = a.row_seq[tok];
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] = TR::store(v[0][i]);
      memcpy((T*)a.vc + ((size_t)(b * a.n_kv + head) * a.max_len + pos) * a.hd + dim, out, sizeof(out));
    }
  }
}

template <int DT, int NT, int MTT, int EPI>
__global__ __launch_bounds__(kWaves * 64) void k_gemm(GemmArgs a) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  constexpr int KT = TR::KT, VEC = TR::VEC;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int ksteps = a.K / KT;
  const int s0 = (w * ksteps) / kWaves, s1 = ((w + 1) * ksteps) / kWaves;
  const int tok0 = blockIdx.x * (MTT * 16);
  const int tile0 = blockIdx.y * NT;

  // bf16 models multiply each weight tile by both operand planes (hi, lo).
  constexpr int PL = DT == RV_BF16 ? 2 : 1;
  const uint4* wp = (const uint4*)a.W + (size_t)tile0 * ksteps * 64 + lane;
  const uint4* xp[PL][MTT];
#pragma unroll
  for (int pl = 0; pl < PL; ++pl)
#pragma unroll
    for (int mt = 0; mt < MTT; ++mt)
      xp[pl][mt] = (const uint4*)((const T*)(pl ? a.X2 : a.X) + (size_t)(tok0 + mt * 16 + (lane & 15)) * a.ldx +
                                  (lane >> 4) * VEC);

  f32x4_t acc[NT][MTT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < MTT; ++mt) acc[nt][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

#pragma unroll 4
  for (int s = s0; s < s1; ++s) {
    uint4 av[NT], bv[PL][MTT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) av[nt] = wp[((size_t)nt * ksteps + s) * 64];
#pragma unroll
    for (int pl = 0; pl < PL; ++pl)
#pragma unroll
      for (int mt = 0; mt < MTT; ++mt) bv[pl][mt] = xp[pl][mt][(size_t)s * (KT / VEC)];
#pragma unroll
    for (int pl = 0; pl < PL; ++pl)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < MTT; ++mt) mma_step<DT>(av[nt], bv[pl][mt], acc[nt][mt]);
  }

  __shared__ f32x4_t red[kWaves][NT][MTT][64];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < MTT; ++mt) red[w][nt][mt][lane] = acc[nt][mt];
  __syncthreads();
  if (w < MTT) {
    const int mt = w;
    f32x4_t v[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      v[nt] = red[0][nt][mt][lane];
#pragma unroll
      for (int ww = 1; ww < kWaves; ++ww) v[nt] += red[ww][nt][mt][lane];
    }
    epilogue<DT, NT, EPI>(a, tile0, tok0 + mt * 16 + (lane & 15), lane, v);
  }
}

template <int DT, int NT, int EPI>
hipError_t launch_mtt(const GemmArgs& a, hipStream_t st) {
  const int rows_per_wg = 16 * NT;
  dim3 block(kWaves * 64);
  if (a.M <= 16) {
    k_gemm<DT, NT, 1, EPI><<<dim3(1, a.N / rows_per_wg), block, 0, st>>>(a);
  } else if (a.M <= 32) {
    k_gemm<DT, NT, 2, EPI><<<dim3(1, a.N / rows_per_wg), block, 0, st>>>(a);
  } else {
    k_gemm<DT, NT, 4, EPI><<<dim3((a.M + 63) / 64, a.N / rows_per_wg), block, 0, st>>>(a);
  }
  return hipGetLastError();
}

template <int DT>
hipError_t launch_dt(int epi, const GemmArgs& a, hipStream_t st) {
  switch (epi) {
    case EPI_STORE: return launch_mtt<DT, 1, EPI_STORE>(a, st);
    case EPI_RESID: return launch_mtt<DT, 1, EPI_RESID>(a, st);
    case EPI_SWIGLU: return launch_mtt<DT, 2, EPI_SWIGLU>(a, st);
    case EPI_QKV: return launch_mtt<DT, 1, EPI_QKV>(a, st);
    case EPI_STORE_LOGICAL: return launch_mtt<DT, 1, EPI_STORE_LOGICAL>(a, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace

// Operand rows read: round_up(M, 16) for M <= 32, else round_up(M, 64); the
// caller's X buffer must hold that many rows.
hipError_t launch_gemm(int dtype, int epi, const GemmArgs& a, hipStream_t st) {
  return dtype == RV_BF16 ? launch_dt<RV_BF16>(epi, a, st) : launch_dt<RV_F32>(epi, a, st);
}
