// Filter banks of the wavelet bases beyond Haar, for the temporal allocator
// (Sec. 3.2.3, Eq. (9)-(11)) and the spatial modulator (Sec. 3.2.3,
// Eq. (12)-(15)): db4, the paper's spatial default (Sec. 4.1), and bior4.4,
// the third basis of its ablation (Sec. 4.3).
//
// Low-pass filters, normalised to sum sqrt(2):
//   db4:     Daubechies' minimum-phase filter with four vanishing moments
//            (I. Daubechies, Ten Lectures on Wavelets, 1992, Table 6.1, N = 4);
//            synthesis h, analysis h reversed;
//   bior4.4: the Cohen-Daubechies-Feauveau 9/7 pair of JPEG 2000's
//            irreversible transform (ISO/IEC 15444-1, Annex F): analysis
//            9 taps, synthesis 7 taps, both placed in 10 with one leading
//            zero.
// High-pass filters: rec_hi[k] = (-1)^k dec_lo[k], dec_hi[k] = -(-1)^k rec_lo[k].
// Conventions of one analysis step on L samples (F taps): half-sample
// symmetric extension x~, n = floor((L + F - 1) / 2) coefficients
//   a[k] = sum_j dec_lo[j] x~[2k + 1 - j]   (d likewise with dec_hi);
// synthesis x[i] = sum_k rec_lo[i + F - 2 - 2k] a[k] + rec_hi[...] d[k],
// cropped to L.  A gate is pooled to a subband's length n by adaptive
// average pooling: output i averages inputs floor(i L / n) ..
// ceil((i + 1) L / n) - 1.
#pragma once

#include "wz_internal.h"

namespace wz {

constexpr int kMaxTaps = 10;

struct Bank {
  int F;  // taps (even)
  double dec_lo[kMaxTaps], dec_hi[kMaxTaps], rec_lo[kMaxTaps], rec_hi[kMaxTaps];
};

// The bank of a wz_basis value other than WZ_HAAR (host and device).
__host__ __device__ inline Bank make_bank(int basis) {
  constexpr double kDb4[8] = {0.2303778133088964, 0.7148465705529154, 0.6308807679298587,  -0.0279837694168599,
                              -0.1870348117190931, 0.0308413818355607, 0.0328830116668852, -0.0105974017850690};
  // JPEG 2000 9/7 low-passes from the centre out (analysis at DC gain 1,
  // synthesis at DC gain 2), rescaled below to sum sqrt(2)
  constexpr double kAna[5] = {0.6029490182363579, 0.2668641184428723, -0.07822326652898785, -0.01686411844287495,
                              0.02674875741080976};
  constexpr double kSyn[4] = {1.115087052456994, 0.5912717631142470, -0.05754352622849957, -0.09127176311424948};
  constexpr double kSqrt2 = 1.4142135623730951;
  Bank b{};
  if (basis == WZ_DB4) {
    b.F = 8;
    for (int k = 0; k < 8; ++k) {
      b.rec_lo[k] = kDb4[k];
      b.dec_lo[k] = kDb4[7 - k];
    }
  } else {  // WZ_BIOR44
    b.F = 10;
    for (int k = 0; k < 10; ++k) b.dec_lo[k] = b.rec_lo[k] = 0.0;
    for (int k = -4; k <= 4; ++k) b.dec_lo[5 + k] = kAna[k < 0 ? -k : k] * kSqrt2;
    for (int k = -3; k <= 3; ++k) b.rec_lo[4 + k] = kSyn[k < 0 ? -k : k] / kSqrt2;
  }
  for (int k = 0; k < b.F; ++k) {
    const double s = (k & 1) ? -1.0 : 1.0;
    b.rec_hi[k] = s * b.dec_lo[k];
    b.dec_hi[k] = -s * b.rec_lo[k];
  }
  return b;
}

// Position of sample i of the half-sample symmetric extension of L samples
// (reflections about -1/2 and L - 1/2; more than one only when L is shorter
// than the filter).
__host__ __device__ inline int sym_index(int i, int L) {
  while (i < 0 || i >= L) i = i < 0 ? -1 - i : 2 * L - 1 - i;
  return i;
}

// Analysis coefficients per band for L samples.
__host__ __device__ inline int bank_len(int L, int F) { return (L + F - 1) / 2; }

}  // namespace wz
