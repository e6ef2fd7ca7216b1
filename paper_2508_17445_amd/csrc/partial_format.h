// Block floating-point storage of partial O rows (plans with compact partial
// slots): a lane's d-group of four fp32 values x_0..x_3 in one 64-bit word.
//   E    the group's largest fp32 exponent field (8 bits): its low nibble in
//        bits 28-31 of word 0, its high nibble in bits 28-31 of word 1;
//   m_k  round(x_k 2^(139 - E)) as a 14-bit two's-complement integer (every
//        |x_k| < 2^(E - 126), so |m_k| <= 8192; clamped to 8191): m_0 and m_1
//        in bits 0-13 and 14-27 of word 0, m_2 and m_3 in word 1;
//   x_k = m_k 2^(E - 139).
// Groups whose E is below 13 (every value under 2^-114) store zeros.  Each
// value is off by at most 2^-13 of its group's largest magnitude.  A group
// holding an infinity or a NaN (E = 255) is stored as E = 255 with zero
// mantissas and decodes to four NaNs, so non-finite partials stay
// non-finite.
#ifndef TREEPO_PARTIAL_FORMAT_H
#define TREEPO_PARTIAL_FORMAT_H

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace treepo {

__host__ __device__ inline uint32_t fp32_bits(float x) { return __builtin_bit_cast(uint32_t, x); }

__host__ __device__ inline int32_t group_mantissa(float x, float scale) {
  const int32_t m = static_cast<int32_t>(rintf(x * scale));
  return m > 8191 ? 8191 : m;
}

__host__ __device__ inline void pack_group4(float x0, float x1, float x2, float x3, uint32_t* w0, uint32_t* w1) {
  const uint32_t e0 = (fp32_bits(x0) >> 23) & 0xFFu, e1 = (fp32_bits(x1) >> 23) & 0xFFu;
  const uint32_t e2 = (fp32_bits(x2) >> 23) & 0xFFu, e3 = (fp32_bits(x3) >> 23) & 0xFFu;
  const uint32_t ea = e0 > e1 ? e0 : e1, eb = e2 > e3 ? e2 : e3;
  const uint32_t e = ea > eb ? ea : eb;
  int32_t m0 = 0, m1 = 0, m2 = 0, m3 = 0;
  if (e >= 13 && e < 255) {
    const float sc = __builtin_bit_cast(float, (266u - e) << 23);  // 2^(139 - E)
    m0 = group_mantissa(x0, sc);
    m1 = group_mantissa(x1, sc);
    m2 = group_mantissa(x2, sc);
    m3 = group_mantissa(x3, sc);
  }
  *w0 = (static_cast<uint32_t>(m0) & 0x3FFFu) | ((static_cast<uint32_t>(m1) & 0x3FFFu) << 14) | (e << 28);
  *w1 = (static_cast<uint32_t>(m2) & 0x3FFFu) | ((static_cast<uint32_t>(m3) & 0x3FFFu) << 14) | ((e >> 4) << 28);
}

__host__ __device__ inline void unpack_group4(uint32_t w0, uint32_t w1, float* f) {
  const uint32_t e = (w0 >> 28) | ((w1 >> 28) << 4);
  // 2^(E - 139); NaN for a non-finite group
  const float sc = e == 255 ? __builtin_bit_cast(float, 0x7FC00000u)
                            : (e >= 13 ? __builtin_bit_cast(float, (e - 12) << 23) : 0.f);
  f[0] = static_cast<float>(static_cast<int32_t>(w0 << 18) >> 18) * sc;
  f[1] = static_cast<float>(static_cast<int32_t>(w0 << 4) >> 18) * sc;
  f[2] = static_cast<float>(static_cast<int32_t>(w1 << 18) >> 18) * sc;
  f[3] = static_cast<float>(static_cast<int32_t>(w1 << 4) >> 18) * sc;
}

}  // namespace treepo

#endif
