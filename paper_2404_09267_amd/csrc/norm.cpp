// Host-side normalisation constants of tg_stitch: the correctly rounded binary16 table
// and the search for exact fp32 fma constants (see norm.h).
#include "norm.h"

#include <cfloat>
#include <cmath>
#include <cstdlib>
#include <cstring>

#include "tg.h"

namespace tg_detail {

// From the double's fields: 1 sign, 11 exponent (bias 1023), 52 fraction bits.
uint16_t half_bits_rne(double v) {
  uint64_t b;
  std::memcpy(&b, &v, sizeof b);
  const uint16_t sign = static_cast<uint16_t>((b >> 48) & 0x8000u);
  const int biased = static_cast<int>((b >> 52) & 0x7FFu);
  const uint64_t frac = b & ((uint64_t(1) << 52) - 1);
  if (biased == 0x7FF) return sign | (frac ? 0x7E00u : 0x7C00u);
  if (biased == 0) return sign;  // below 2^-1022: far under half's smallest subnormal
  const int e = biased - 1023;
  if (e > 15) return sign | 0x7C00u;
  const uint64_t sig = frac | (uint64_t(1) << 52);  // value = sig * 2^(e - 52)
  // Normal halves keep 10 fraction bits (drop 42); subnormals count units of 2^-24.
  const int drop = e >= -14 ? 42 : 28 - e;
  if (drop > 53) return sign;  // below 2^-25: rounds to zero
  uint64_t q = sig >> drop;
  const uint64_t rest = sig & ((uint64_t(1) << drop) - 1);
  const uint64_t halfway = uint64_t(1) << (drop - 1);
  if (rest > halfway || (rest == halfway && (q & 1))) ++q;
  // Normal: exponent field (e + 15) plus q - 1024; a carry to q == 2048 bumps the
  // exponent (and at e == 15 lands exactly on infinity). Subnormal: q itself, where
  // q == 1024 is the smallest normal's encoding.
  const uint32_t bits = e >= -14 ? (uint32_t(e + 15) << 10) + uint32_t(q - 1024) : uint32_t(q);
  return static_cast<uint16_t>(sign | bits);
}

namespace {

float step_ulps(float v, int d) {
  for (; d > 0; --d) v = std::nextafter(v, INFINITY);
  for (; d < 0; ++d) v = std::nextafter(v, -INFINITY);
  return v;
}

// Finite and either zero or normal: no denormal operand or result, so the kernel's
// result does not depend on the denormal mode.
bool usable(float v) { return std::isfinite(v) && (v == 0.0f || std::fabs(v) >= FLT_MIN); }

// An fp32 pair (a, c) with binary16(fma(x, a, c)) == want[x] for every byte x, whether
// the fma is rounded once to binary16 or first to fp32; searched among a few ulps
// around (1/std, -mean/std), nearest first.
bool exact_affine(double mean, double stdv, const uint16_t *want, float &a_out, float &c_out) {
  const float a0 = static_cast<float>(1.0 / stdv), c0 = static_cast<float>(-mean / stdv);
  for (int d = 0; d <= 6; ++d)
    for (int da = -d; da <= d; ++da)
      for (int dc = -d; dc <= d; ++dc) {
        if (std::abs(da) != d && std::abs(dc) != d) continue;
        const float a = step_ulps(a0, da), c = step_ulps(c0, dc);
        if (!usable(a) || !usable(c)) continue;
        bool ok = true;
        for (int x = 0; x < 256 && ok; ++x) {
          const float y = std::fma(static_cast<float>(x), a, c);  // through fp32
          ok = usable(y) && half_bits_rne(static_cast<double>(y)) == want[x];
          // once: x * a is exact in double; the sum's rounding error e (two-sum) must
          // not be able to move it across a binary16 rounding boundary
          const double p = static_cast<double>(x) * static_cast<double>(a);
          const double q = p + static_cast<double>(c);
          const double bp = q - p, e = (p - (q - bp)) + (static_cast<double>(c) - bp);
          ok = ok && half_bits_rne(q) == want[x];
          if (ok && e != 0.0)
            ok = half_bits_rne(std::nextafter(q, -INFINITY)) == want[x] &&
                 half_bits_rne(std::nextafter(q, INFINITY)) == want[x];
        }
        if (ok) {
          a_out = a;
          c_out = c;
          return true;
        }
      }
  return false;
}

}  // namespace

const NormConsts &norm_consts(const float mean[3], const float stdv[3]) {
  thread_local NormConsts cache;
  thread_local bool valid = false;
  if (valid && std::memcmp(cache.mean, mean, sizeof cache.mean) == 0 &&
      std::memcmp(cache.std, stdv, sizeof cache.std) == 0)
    return cache;
  std::memcpy(cache.mean, mean, sizeof cache.mean);
  std::memcpy(cache.std, stdv, sizeof cache.std);
  for (int k = 0; k < 3; ++k)
    for (int x = 0; x < 256; ++x)
      cache.lut16[k * 256 + x] = half_bits_rne((double(x) - double(mean[k])) / double(stdv[k]));
  cache.affine = true;
  for (int k = 0; k < 3; ++k) {
    cache.fa[k] = cache.fc[k] = 0.0f;
    if (cache.affine)
      cache.affine =
          exact_affine(mean[k], stdv[k], cache.lut16 + 256 * k, cache.fa[k], cache.fc[k]);
  }
  valid = true;
  return cache;
}

}  // namespace tg_detail

extern "C" int32_t tg_stitch_norm_uses_table(const float mean[3], const float stdv[3]) {
  if (!mean || !stdv) return TG_E_INVAL;
  for (int k = 0; k < 3; ++k)
    if (!std::isfinite(mean[k]) || !std::isfinite(stdv[k]) || !(stdv[k] > 0.0f))
      return TG_E_INVAL;
  return tg_detail::norm_consts(mean, stdv).affine ? 0 : 1;
}
