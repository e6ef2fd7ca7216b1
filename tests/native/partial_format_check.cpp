// Host check of the block floating-point partial-row format
// (paper_2508_17445_amd/csrc/partial_format.h): the documented bit layout on
// hand-worked groups, and the error bound -- every decoded value within 2^-13
// of its group's largest magnitude -- on random groups spanning the fp32
// exponent range, with sign mixes, zeros and values 2^-20 below the maximum;
// groups holding an infinity or a NaN decode to NaNs.
// Prints "ok <worst relative error>" or the first failure.
#include <math.h>
#include <stdio.h>
#include <stdint.h>

#include <random>

#include "partial_format.h"

using treepo::pack_group4;
using treepo::unpack_group4;

static int check_exact(float x0, float x1, float x2, float x3, uint32_t w0, uint32_t w1) {
  uint32_t a, b;
  pack_group4(x0, x1, x2, x3, &a, &b);
  if (a != w0 || b != w1) {
    printf("layout (%g %g %g %g): %08x %08x, expected %08x %08x\n", x0, x1, x2, x3, a, b, w0, w1);
    return 1;
  }
  float f[4];
  unpack_group4(a, b, f);
  const float x[4] = {x0, x1, x2, x3};
  for (int k = 0; k < 4; ++k)
    if (f[k] != x[k]) {
      printf("decode (%g %g %g %g)[%d] = %g\n", x0, x1, x2, x3, k, f[k]);
      return 1;
    }
  return 0;
}

int main() {
  // E = 127 (1.0): m = x * 2^12; 1.0 -> 4096, -1.0 -> -4096 (0x3000 in 14
  // bits), 0.5 -> 2048; E's nibbles 0xF and 0x7 in bits 28-31.
  if (check_exact(1.0f, -1.0f, 0.5f, 0.0f, 0x1000u | (0x3000u << 14) | (0xFu << 28), 0x800u | (0x7u << 28)))
    return 1;
  // E = 130 (|x| in [8, 16)): m = x * 2^9; -12.5 -> -6400 (0x2700), 3 -> 1536
  if (check_exact(3.0f, -12.5f, 0.0f, 8.0f, 1536u | (0x2700u << 14) | (0x2u << 28), (4096u << 14) | (0x8u << 28)))
    return 1;
  // all zeros, and a group below 2^-114, store zeros (E < 13 keeps its nibbles)
  if (check_exact(0.0f, 0.0f, 0.0f, 0.0f, 0u, 0u)) return 1;
  // a group holding an infinity or a NaN: E = 255, zero mantissas, four NaNs
  {
    const float bad[3] = {INFINITY, -INFINITY, NAN};
    for (int i = 0; i < 3; ++i)
      for (int k = 0; k < 4; ++k) {
        float x[4] = {1.0f, -2.0f, 0.25f, 0.0f};
        x[k] = bad[i];
        uint32_t a, b;
        pack_group4(x[0], x[1], x[2], x[3], &a, &b);
        if (a != (0xFu << 28) || b != (0xFu << 28)) {
          printf("non-finite group %d/%d: %08x %08x\n", i, k, a, b);
          return 1;
        }
        float f[4];
        unpack_group4(a, b, f);
        for (int j = 0; j < 4; ++j)
          if (!isnan(f[j])) {
            printf("non-finite group %d/%d decodes to %g at %d\n", i, k, f[j], j);
            return 1;
          }
      }
  }
  std::mt19937 g(7);
  std::normal_distribution<float> n(0.f, 1.f);
  std::uniform_real_distribution<float> u(-100.f, 100.f), v(-20.f, 0.f);
  double worst = 0.0;
  for (int t = 0; t < 2000000; ++t) {
    const float s = ldexpf(1.0f, static_cast<int>(u(g)));
    float x[4];
    for (int k = 0; k < 4; ++k) x[k] = n(g) * s * ldexpf(1.0f, static_cast<int>(v(g)));
    if (t % 7 == 0) x[t % 4] = 0.0f;
    uint32_t a, b;
    pack_group4(x[0], x[1], x[2], x[3], &a, &b);
    float f[4];
    unpack_group4(a, b, f);
    double mx = 0.0, err = 0.0;
    for (int k = 0; k < 4; ++k) mx = fmax(mx, fabs(static_cast<double>(x[k])));
    for (int k = 0; k < 4; ++k) err = fmax(err, fabs(static_cast<double>(f[k]) - static_cast<double>(x[k])));
    if (mx < ldexp(1.0, -110)) {
      if (err > ldexp(1.0, -110)) {
        printf("tiny group error %g\n", err);
        return 1;
      }
      continue;
    }
    const double rel = err / mx;
    if (rel > worst) worst = rel;
    if (rel > ldexp(1.0, -13)) {
      printf("bound (%g %g %g %g) -> (%g %g %g %g): %g of the group maximum\n", x[0], x[1], x[2], x[3], f[0],
             f[1], f[2], f[3], rel);
      return 1;
    }
  }
  printf("ok %.6g\n", worst);
  return 0;
}
