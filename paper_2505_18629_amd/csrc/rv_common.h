// Shared device definitions of the gfx950 verify-pass library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include "rv.h"

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

#define RV_DEV __device__ __forceinline__

// ---------------------------------------------------------------- rounding

// fp32 -> bf16 bits, round to nearest even (gfx950 converts in hardware,
// v_cvt_pk_bf16_f32; denormals are kept and NaN stays NaN).
RV_DEV uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
RV_DEV float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Storage type traits: weights, matmul operands and KV are T; a k-step of
// the matrix kernels consumes one 1 KiB tile of 16 rows x KT elements, in
// which lane l holds row l % 16 and the VEC consecutive k elements starting
// at (l / 16) * VEC.
template <int DT> struct Tr;
template <> struct Tr<RV_BF16> {
  typedef uint16_t T;
  static constexpr int KT = 32, VEC = 8;
  static RV_DEV T store(float x) { return f2bf(x); }
  static RV_DEV float load(T x) { return bf2f(x); }
};
template <> struct Tr<RV_F32> {
  typedef float T;
  static constexpr int KT = 16, VEC = 4;
  static RV_DEV T store(float x) { return x; }
  static RV_DEV float load(T x) { return x; }
};

// One k-step of a 16x16 output tile: acc += A(16 x KT) . B(KT x 16), with A
// and B given as the 16 bytes each lane holds.  Hardware k slots of lane
// group g are mapped to logical k = g * VEC + j for both operands, so the
// reduction covers exactly the tile's KT elements.
template <int DT> RV_DEV void mma_step(const uint4& a, const uint4& b, f32x4_t& acc);
template <> RV_DEV void mma_step<RV_BF16>(const uint4& a, const uint4& b, f32x4_t& acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}
template <> RV_DEV void mma_step<RV_F32>(const uint4& a, const uint4& b, f32x4_t& acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// Operand form of an fp32 activation that feeds a matmul.  bf16 models keep
// two planes, hi = bf16(x) and lo = bf16(x - hi) (x - hi is exact in fp32),
// so an operand carries ~16 significant bits and a matmul is two MFMAs;
// fp32 models keep x in the first plane.
//
// Operand planes are stored in MFMA B-operand tiles, the same 1 KiB tiling
// as the packed weights with tokens in place of output rows: tile
// (token/16, k/KT), lane (token%16) + 16*((k%KT)/VEC), VEC elements per lane.
// A matmul wave reads one tile with one contiguous 16-byte load per lane.
RV_DEV __host__ inline size_t operand_offset(int t, int k, int K, int es) {
  const int vec = 16 / es, kt = 4 * vec;
  const int kin = k % kt;
  return (((size_t)(t >> 4) * (K / kt) + k / kt) * 64 + (t & 15) + 16 * (kin / vec)) * 16 + (size_t)(kin % vec) * es;
}

// Stores x (4 consecutive k, k % 4 == 0) of token t into the operand planes.
template <int DT> RV_DEV void put_operand4(void* hi, void* lo, int t, int k, int K, const f32x4_t& x);
template <> RV_DEV void put_operand4<RV_BF16>(void* hi, void* lo, int t, int k, int K, const f32x4_t& x) {
  uint16_t h[4], l[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    h[j] = f2bf(x[j]);
    l[j] = f2bf(x[j] - bf2f(h[j]));
  }
  const size_t o = operand_offset(t, k, K, 2);
  memcpy((char*)hi + o, h, 8);
  memcpy((char*)lo + o, l, 8);
}
template <> RV_DEV void put_operand4<RV_F32>(void* hi, void*, int t, int k, int K, const f32x4_t& x) {
  memcpy((char*)hi + operand_offset(t, k, K, 4), &x, 16);
}

// K/V cache.  Each (sequence, kv head) owns kv_len positions (a multiple of
// 64) of hd values.  fp32 models store them row-major.  bf16 models store hi
// and lo planes in the order the attention MFMAs consume them, so that a
// 64-key tile is one contiguous span per plane and every operand is one
// 16-byte LDS read per lane:
//  K: 16-position blocks; unit (block, 32-dim chunk c) is 1 KiB, lane l
//     holding positions 16*block + l%16, dims 32c + 8*(l/16) .. +7 (the A
//     operand of S^T = K Q^T).
//  V: 32-position blocks; unit (block, 16-dim tile t) is 1 KiB, lane l
//     holding dim 16t + l%16 of the 8 keys of slot group g = l/16: keys
//     4g..4g+3 and 16+4g..16+4g+3 of the block (the A operand of
//     O^T += V^T P^T, whose B operand comes straight from the score
//     registers in that key order).
RV_DEV __host__ inline size_t k_elem(int pos, int d, int hd) {
  return ((size_t)(pos >> 4) * (hd >> 5) + (d >> 5)) * 512 + ((pos & 15) + 16 * ((d & 31) >> 3)) * 8 + (d & 7);
}
RV_DEV __host__ inline size_t v_elem(int pos, int d, int hd) {
  const int kk = pos & 31;
  return ((size_t)(pos >> 5) * (hd >> 4) + (d >> 4)) * 512 + ((d & 15) + 16 * ((kk & 15) >> 2)) * 8 + (kk & 3) +
         4 * (kk >> 4);
}

// Stores x = dims d..d+3 (d % 4 == 0) of position pos into the K or V cache
// block starting at element `base`.
template <int DT> RV_DEV void put_k4(void* hi, void* lo, size_t base, int pos, int d, int hd, const f32x4_t& x);
template <int DT> RV_DEV void put_v4(void* hi, void* lo, size_t base, int pos, int d, int hd, const f32x4_t& x);
template <>
RV_DEV void put_k4<RV_BF16>(void* hi, void* lo, size_t base, int pos, int d, int hd, const f32x4_t& x) {
  uint16_t h[4], l[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    h[j] = f2bf(x[j]);
    l[j] = f2bf(x[j] - bf2f(h[j]));
  }
  const size_t i = base + k_elem(pos, d, hd);  // the 4 dims are adjacent
  memcpy((uint16_t*)hi + i, h, 8);
  memcpy((uint16_t*)lo + i, l, 8);
}
template <>
RV_DEV void put_v4<RV_BF16>(void* hi, void* lo, size_t base, int pos, int d, int hd, const f32x4_t& x) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint16_t h = f2bf(x[j]);
    const size_t i = base + v_elem(pos, d + j, hd);  // 8 elements apart
    ((uint16_t*)hi)[i] = h;
    ((uint16_t*)lo)[i] = f2bf(x[j] - bf2f(h));
  }
}
template <>
RV_DEV void put_k4<RV_F32>(void* hi, void*, size_t base, int pos, int d, int hd, const f32x4_t& x) {
  memcpy((float*)hi + base + (size_t)pos * hd + d, &x, 16);
}
template <>
RV_DEV void put_v4<RV_F32>(void* hi, void*, size_t base, int pos, int d, int hd, const f32x4_t& x) {
  memcpy((float*)hi + base + (size_t)pos * hd + d, &x, 16);
}

// ---------------------------------------------------------------- packing

// Kinds of stored (fused) matrices.  Physical row order differs from the
// logical one so that each 16-row tile carries what its epilogue needs:
//  QKV:    per q/k head, tile j holds dims 8j..8j+7 (rows 0..7) and their
//          rotate-half partners hd/2+8j.. (rows 8..15); v rows are in order.
//  GATEUP: tile 2t holds gate rows 16t..16t+15, tile 2t+1 the same up rows.
enum MatKind { MAT_PLAIN = 0, MAT_QKV = 1, MAT_GATEUP = 2 };

struct MatDesc {
  int kind;
  int N, K;                    // physical rows (= logical rows), reduction length
  int hd, q_rows, k_rows;      // QKV: head_dim, Hq*hd, Hkv*hd
};

// Logical row of fused-matrix physical row p.
RV_DEV __host__ inline int mat_logical_row(const MatDesc& m, int p) {
  if (m.kind == MAT_GATEUP) {
    int tile = p >> 4, r = p & 15;
    int half = m.N / 2;
    return (tile & 1) * half + (tile >> 1) * 16 + r;
  }
  if (m.kind == MAT_QKV && p < m.q_rows + m.k_rows) {
    int head = p / m.hd, within = p % m.hd;
    int j = within >> 4, r = within & 15;
    int dim = r < 8 ? 8 * j + r : m.hd / 2 + 8 * j + (r - 8);
    return head * m.hd + dim;
  }
  return p;
}

// Byte offset of packed element (physical row p, k) for element size es.
RV_DEV __host__ inline size_t mat_packed_offset(const MatDesc& m, int p, int k, int es) {
  int vec = 16 / es, kt = 4 * vec;
  int ksteps = m.K / kt;
  int tile_k = k / kt, kin = k % kt;
  int lane = (p & 15) + 16 * (kin / vec);
  int j = kin % vec;
  return (((size_t)(p >> 4) * ksteps + tile_k) * 1024) + (size_t)lane * 16 + (size_t)j * es;
}

// ---------------------------------------------------------------- reductions

// Reductions over the four lanes that share l % 16 (l, l^16, l^32, l^48) with
// gfx950's row-swap permutes, which run on the VALU instead of the LDS
// crossbar that a shuffle takes.  Swapping x with itself leaves, in the two
// results, x's own row and the partner row (rows of 16 lanes for the first
// swap, halves of the wave for the second), so each step combines a lane with
// its partner in the same order for every lane of the pair: the results equal
// two xor shuffles (16, then 32).
RV_DEV float rows4_max(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(s[0]), __uint_as_float(s[1]));
}
RV_DEV float rows4_sum(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

RV_DEV float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
RV_DEV float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
