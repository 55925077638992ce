// Host-side normalisation constants of tg_stitch (library-internal).
//
// A source byte x of channel k becomes binary16((x - mean[k]) / std[k]), the quotient
// taken in double and rounded once to nearest-even. The kernel gets both a 3 x 256
// table of those values and, when they exist, fp32 constants (a_k, c_k) such that
// binary16(fma(x, a_k, c_k)) equals the table for all 256 bytes -- whether the fma is
// rounded once to binary16 or first to fp32 -- so that it may compute instead of look up.
#ifndef TG_NORM_H
#define TG_NORM_H

#include <cstdint>

namespace tg_detail {

struct NormConsts {
  float mean[3], std[3];
  bool affine;     // fa/fc valid for all three channels
  float fa[3], fc[3];
  uint16_t lut16[768];  // channel k, byte x at k * 256 + x
};

// Constants for (mean, std); the last result is cached per host thread.
const NormConsts &norm_consts(const float mean[3], const float stdv[3]);

// Correctly rounded binary16 of a double (round to nearest, ties to even).
uint16_t half_bits_rne(double v);

}  // namespace tg_detail

#endif  // TG_NORM_H
