/*
 * oracle/weights.c -- TEST INFRASTRUCTURE ONLY.
 *
 * Seeded weight generator for the CPU oracle. Only tests/, the smoke check
 * and the benchmark's CPU-baseline leg may load this library; the product
 * path never does.
 *
 * The paper evaluates trained Llama-3 models (Section 4.1); no weights are
 * available here, so both the oracle and the GPU library regenerate the same
 * random-init weights from (tensor index, element index, seed) with a
 * counter-based generator.  Each side implements the generator on its own
 * from its published definition:
 *
 *   splitmix64 (Steele, Lea, Flood, "Fast splittable pseudorandom number
 *   generators", OOPSLA 2014): state advances by the golden-ratio constant
 *   0x9E3779B97F4A7C15 and each output is the state passed through the
 *   variant-13 finaliser (xor-shift 30, multiply 0xBF58476D1CE4E5B9,
 *   xor-shift 27, multiply 0x94D049BB133111EB, xor-shift 31).
 *
 * Element (r, c) of a logical W[out][in] has index i = r*in + c.  Its value:
 *   h  = mix(((t << 36) + i) ^ mix(seed))       mix(x) = finaliser(x + golden)
 *   s  = sum of the four 16-bit fields of h - 2*65535   (Irwin-Hall(4), exact)
 *   w  = fp32(s) * c   in fp32, c = fp32(std / sqrt(4 * (65536^2 - 1) / 12))
 *   bf16 tensors store RNE_bf16(w); fp32 tensors store w.
 * Tensor numbering: 0 = token embedding [V][d]; for layer l the seven
 * matrices q, k, v, o, gate, up, down are 1 + 7l + {0..6}; 1 + 7L = LM head.
 * Every step is integer or a single correctly rounded fp32 multiply, so an
 * independent implementation reproduces the bits exactly.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

static uint64_t finalise(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static uint64_t mix(uint64_t x) { return finalise(x + GOLDEN); }

/* The first n outputs of a splitmix64 stream started at `seed`. */
void orc_splitmix64_stream(uint64_t seed, int n, uint64_t* out) {
  uint64_t state = seed;
  for (int j = 0; j < n; ++j) {
    state += GOLDEN;
    out[j] = finalise(state);
  }
}

/* fp32 -> bf16 bits, round to nearest even (finite inputs). */
static uint16_t bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static float bf16_to_f32(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

float orc_scale(double init_std) {
  double sd = sqrt(4.0 * (65536.0 * 65536.0 - 1.0) / 12.0);
  return (float)(init_std / sd);
}

static float element(uint64_t seed_mix, uint64_t t, uint64_t i, float c, int bf16) {
  uint64_t h = mix(((t << 36) + i) ^ seed_mix);
  int32_t s = (int32_t)(h & 0xFFFF) + (int32_t)((h >> 16) & 0xFFFF) +
              (int32_t)((h >> 32) & 0xFFFF) + (int32_t)(h >> 48) - 2 * 65535;
  float w = (float)s * c;
  return bf16 ? bf16_to_f32(bf16_rne(w)) : w;
}

/* Writes logical elements [start, start + count) of tensor t as doubles
 * (the values are exact).  bf16 != 0 selects bf16 rounding. */
void orc_fill(uint64_t seed, uint64_t t, uint64_t start, uint64_t count, int bf16,
              double init_std, double* out) {
  uint64_t sm = mix(seed);
  float c = orc_scale(init_std);
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < (int64_t)count; ++j)
    out[j] = (double)element(sm, t, start + (uint64_t)j, c, bf16);
}

/* Bit pattern of single elements at arbitrary indices (for bit-equality
 * checks of a device buffer): fp32 bits, or bf16 bits in the low half. */
void orc_bits_at(uint64_t seed, uint64_t t, const uint64_t* idx, int64_t n, int bf16,
                 double init_std, uint32_t* out) {
  uint64_t sm = mix(seed);
  float c = orc_scale(init_std);
  for (int64_t j = 0; j < n; ++j) {
    float w = element(sm, t, idx[j], c, 0);
    if (bf16) {
      out[j] = bf16_rne(w);
    } else {
      uint32_t u;
      memcpy(&u, &w, 4);
      out[j] = u;
    }
  }
}

/* Round an array of doubles through fp32 to bf16 (RNE at each step, the
 * path an fp32 kernel value takes when it is stored as bf16). */
void orc_round_bf16(const double* in, double* out, int64_t n) {
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) out[j] = (double)bf16_to_f32(bf16_rne((float)in[j]));
}
