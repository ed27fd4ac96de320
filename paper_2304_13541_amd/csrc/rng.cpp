// Seeded weight generation for random-weight models (the paper evaluates
// trained torchvision models, Sec. 3; here the same architectures carry
// synthetic weights drawn from a seed).
//
// splitmix64 (Steele, Lea, Flood, OOPSLA 2014): state += 0x9E3779B97F4A7C15,
// then two xor-shift-multiply rounds.  Tensor t of seed S starts from
// S ^ (0x9E3779B97F4A7C15 * (t + 1)).  u = (next >> 11) * 2^-53 with 0 -> 1.
// Normals: Box-Muller (Box & Muller 1958) pairs, both outputs in order.
// Every value is rounded to bf16 (round to nearest, ties to even) directly
// from fp64.  Compiled with -ffp-contract=off so that every fp64 operation
// rounds exactly as written.
#include "model.hpp"

#include <cmath>
#include <cstring>

namespace dstack {

namespace {

struct SplitMix64 {
  uint64_t s;
  uint64_t next() {
    s += 0x9E3779B97F4A7C15ULL;
    uint64_t z = s;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
  }
  double unit() {
    uint64_t r = next() >> 11;
    return r == 0 ? 1.0 : (double)r * (1.0 / 9007199254740992.0);
  }
};

}  // namespace

// Round-to-nearest-even of an fp64 value to bf16, on the bit pattern:
// keep 7 of the 52 stored fraction bits (45 dropped), or, below the bf16
// normal range, quantise the full significand to multiples of 2^-133.
uint16_t bf16_from_double(double x) {
  uint64_t u;
  std::memcpy(&u, &x, 8);
  const uint16_t sign = (uint16_t)((u >> 63) << 15);
  const int bexp = (int)((u >> 52) & 0x7FF);
  const uint64_t frac = u & ((1ULL << 52) - 1);
  if (bexp == 0 && frac == 0) return sign;  // +-0 (fp64 subnormals are far below bf16's range)
  if (bexp == 0) return sign;
  const int e = bexp - 1023;
  if (e >= -126) {
    uint64_t keep = frac >> 45;
    const uint64_t rest = frac & ((1ULL << 45) - 1);
    const uint64_t half = 1ULL << 44;
    int ee = e;
    if (rest > half || (rest == half && (keep & 1))) {
      ++keep;
      if (keep == 128) {
        keep = 0;
        ++ee;
      }
    }
    return (uint16_t)(sign | (uint16_t)((ee + 127) << 7) | (uint16_t)keep);
  }
  // bf16 subnormal: value = sig * 2^(e - 52), quantum 2^-133 -> q = sig >> (-81 - e)
  const uint64_t sig = frac | (1ULL << 52);
  const int sh = -81 - e;  // >= 46
  if (sh >= 64) return sign;
  uint64_t q = sig >> sh;
  const uint64_t rest = sig & ((1ULL << sh) - 1);
  const uint64_t half = 1ULL << (sh - 1);
  if (rest > half || (rest == half && (q & 1))) ++q;
  return (uint16_t)(sign | (uint16_t)q);  // q == 128 is the smallest normal, bits 0x0080
}

void generate_tensor(uint64_t seed, int index, const TensorSpec& t, uint16_t* out) {
  SplitMix64 g{seed ^ (0x9E3779B97F4A7C15ULL * (uint64_t)(index + 1))};
  const int64_t n = t.numel;
  if (t.dist == DIST_ZERO) {
    std::memset(out, 0, sizeof(uint16_t) * (size_t)n);
  } else if (t.dist == DIST_HE) {
    const double sd = std::sqrt(2.0 / (double)t.fan_in);
    const double two_pi = 6.283185307179586;
    for (int64_t i = 0; i < n; i += 2) {
      double u1 = g.unit();
      double u2 = g.unit();
      double r = std::sqrt(-2.0 * std::log(u1));
      double th = two_pi * u2;
      double z0 = r * std::cos(th);
      double z1 = r * std::sin(th);
      out[i] = bf16_from_double(z0 * sd);
      if (i + 1 < n) out[i + 1] = bf16_from_double(z1 * sd);
    }
  } else {  // DIST_LSTM: (2u - 1) / 32
    const double a = 1.0 / 32.0;
    for (int64_t i = 0; i < n; ++i) {
      double v = 2.0 * g.unit();
      v = v - 1.0;
      out[i] = bf16_from_double(v * a);
    }
  }
}

}  // namespace dstack
