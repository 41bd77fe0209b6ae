// Seeded random-init weights written directly in the layouts the kernels read.
//
// Generator (device side; the CPU oracle has its own implementation): the
// value of logical element i of tensor t is an Irwin-Hall(4) sum of the four
// 16-bit fields of a splitmix64 hash (Steele, Lea, Flood, OOPSLA 2014) of
// ((t << 36) + i) ^ mix(seed), scaled by an fp32 constant and rounded to the
// storage type.  Only integer operations and one fp32 multiply are involved,
// so the bits are fully determined.
#include "rv_internal.h"

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ULL;

RV_DEV uint64_t sm_finalise(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

RV_DEV float gen_value(uint64_t seed_mix, uint64_t tensor, uint64_t idx, float scale) {
  // h = mix(key ^ mix(seed)) with mix(x) = finalise(x + golden); seed_mix = mix(seed)
  uint64_t hv = sm_finalise((((tensor << 36) + idx) ^ seed_mix) + kGolden);
  int s = (int)(hv & 0xFFFFu) + (int)((hv >> 16) & 0xFFFFu) + (int)((hv >> 32) & 0xFFFFu) +
          (int)(hv >> 48) - 2 * 65535;
  return (float)s * scale;
}

// Source tensor and logical row of a fused matrix's logical row.
struct SrcMap {
  int kind;            // MatKind
  uint64_t t0, t1, t2; // generator tensor ids of the fused parts
  int r1, r2;          // logical-row boundaries of parts 1 and 2
};

RV_DEV void src_of(const SrcMap& s, int lr, uint64_t& t, int& r) {
  if (lr < s.r1) { t = s.t0; r = lr; }
  else if (lr < s.r2) { t = s.t1; r = lr - s.r1; }
  else { t = s.t2; r = lr - s.r2; }
}

// One thread writes one 16-byte packed chunk (lane slot of a 1 KiB tile).
template <int DT>
__global__ void k_init_packed(typename Tr<DT>::T* __restrict__ dst, MatDesc md, SrcMap sm,
                              uint64_t seed_mix, float scale, size_t n_chunks) {
  using TR = Tr<DT>;
  constexpr int VEC = TR::VEC, KT = TR::KT;
  size_t c = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= n_chunks) return;
  size_t tile = c >> 6;
  int lane = (int)(c & 63);
  int ksteps = md.K / KT;
  int p = (int)(tile / ksteps) * 16 + (lane & 15);
  int k0 = (int)(tile % ksteps) * KT + (lane >> 4) * VEC;
  int lr = mat_logical_row(md, p);
  uint64_t t;
  int r;
  src_of(sm, lr, t, r);
  typename TR::T v[VEC];
#pragma unroll
  for (int j = 0; j < VEC; ++j) v[j] = TR::store(gen_value(seed_mix, t, (uint64_t)r * md.K + k0 + j, scale));
  memcpy(dst + c * VEC, v, 16);
}

// Row-major [rows][cols] tensor (embedding).
template <int DT>
__global__ void k_init_rowmajor(typename Tr<DT>::T* __restrict__ dst, uint64_t tensor, uint64_t seed_mix,
                                float scale, size_t n) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  dst[i] = Tr<DT>::store(gen_value(seed_mix, tensor, i, scale));
}

__global__ void k_fill_f32(float* __restrict__ dst, float v, size_t n) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = v;
}

}  // namespace

hipError_t launch_init_packed(int dtype, void* dst, const MatDesc& md, uint64_t t0, uint64_t t1, uint64_t t2,
                              int r1, int r2, uint64_t seed_mix, float scale, hipStream_t st) {
  SrcMap sm{md.kind, t0, t1, t2, r1, r2};
  int es = dtype == RV_BF16 ? 2 : 4;
  size_t n_chunks = (size_t)md.N * md.K * es / 16;
  dim3 grid((unsigned)((n_chunks + 255) / 256));
  if (dtype == RV_BF16)
    k_init_packed<RV_BF16><<<grid, 256, 0, st>>>((uint16_t*)dst, md, sm, seed_mix, scale, n_chunks);
  else
    k_init_packed<RV_F32><<<grid, 256, 0, st>>>((float*)dst, md, sm, seed_mix, scale, n_chunks);
  return hipGetLastError();
}

hipError_t launch_init_rowmajor(int dtype, void* dst, uint64_t tensor, size_t n, uint64_t seed_mix, float scale,
                                hipStream_t st) {
  dim3 grid((unsigned)((n + 255) / 256));
  if (dtype == RV_BF16)
    k_init_rowmajor<RV_BF16><<<grid, 256, 0, st>>>((uint16_t*)dst, tensor, seed_mix, scale, n);
  else
    k_init_rowmajor<RV_F32><<<grid, 256, 0, st>>>((float*)dst, tensor, seed_mix, scale, n);
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* dst, float v, size_t n, hipStream_t st) {
  k_fill_f32<<<dim3((unsigned)((n + 255) / 256)), 256, 0, st>>>(dst, v, n);
  return hipGetLastError();
}
