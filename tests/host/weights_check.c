/* The oracle's weight generator (oracle/weights.c) built with the address
 * and undefined-behaviour sanitizers and driven over the index ranges the
 * workloads use (the largest tensor index and flat element index of the 70B
 * shape included): prints one line of values per call so that
 * tests/test_host_checks.py can compare them with the normally built
 * library the oracle loads. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void orc_splitmix64_stream(uint64_t seed, int n, uint64_t* out);
float orc_scale(double init_std);
void orc_fill(uint64_t seed, uint64_t t, uint64_t start, uint64_t count, int bf16, double init_std, double* out);
void orc_bits_at(uint64_t seed, uint64_t t, const uint64_t* idx, int64_t n, int bf16, double init_std,
                 uint32_t* out);
void orc_round_bf16(const double* in, double* out, int64_t n);

int main(void) {
  uint64_t st[4];
  orc_splitmix64_stream(0, 4, st);
  printf("stream %llu %llu %llu %llu\n", (unsigned long long)st[0], (unsigned long long)st[1],
         (unsigned long long)st[2], (unsigned long long)st[3]);
  /* (tensor, start) pairs: the embedding, a layer matrix, the 70B LM head
   * (tensor 1 + 7 * 80) at its last elements (128256 x 8192) */
  const uint64_t cases[4][2] = {{0, 0}, {9, 123456789}, {561, 128256ull * 8192 - 16}, {561, 0}};
  double v[16];
  for (int c = 0; c < 4; ++c) {
    for (int bf16 = 0; bf16 < 2; ++bf16) {
      orc_fill(7, cases[c][0], cases[c][1], 16, bf16, 0.02, v);
      printf("fill %llu %llu %d", (unsigned long long)cases[c][0], (unsigned long long)cases[c][1], bf16);
      for (int j = 0; j < 16; ++j) printf(" %.17g", v[j]);
      printf("\n");
    }
  }
  uint64_t idx[3] = {0, 5, 128256ull * 8192 - 1};
  uint32_t bits[3];
  orc_bits_at(7, 561, idx, 3, 1, 0.02, bits);
  printf("bits %u %u %u\n", bits[0], bits[1], bits[2]);
  double in[4] = {1.0 + 1.0 / 256, -3.0000001, 1e-40, 65504.5}, out[4];
  orc_round_bf16(in, out, 4);
  printf("round %.17g %.17g %.17g %.17g\n", out[0], out[1], out[2], out[3]);
  return 0;
}
