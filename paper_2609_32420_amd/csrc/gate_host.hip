// Compatibility gate of a recalled cache: host code (a handful of objects and
// candidates per request, decided before any denoising work is issued).
//
// Sec. 3.2 ("Reuse Validity with Generation-Native Evidence"): per object the
// Early Signature holds the normalised support size A (mean of the binary
// tail-frame mask), the mask and a CIELAB colour; against a candidate,
// d_size = |ln(A_q / A_j)|, d_shape = 1 - Dice of the masks cropped to their
// bounding boxes and resampled to a common grid, d_color = CIEDE2000; a
// candidate passes when every discrepancy is within its threshold, and the
// first passing candidate in recall order is reused ("Compatibility
// Filtering").  Sec. 3.2 ("Risk-Aware Compatibility Decisions") and Appendix
// F certify thresholds with the one-sided Clopper-Pearson upper bound.
//
// CIEDE2000: Sharma, Wu and Dalal (2005), kL = kC = kH = 1.  The bound: the p
// at which the binomial probability of at most u failures in n trials equals
// alpha, found by bisection on p (the tail decreases in p), the tail summed
// in log space.
#include "internal.h"

#include <math.h>

namespace carnator {
namespace {

constexpr double kPi = 3.14159265358979323846;
inline double rad(double deg) { return deg * (kPi / 180.0); }

}  // namespace

double ciede2000_pair(const double *x, const double *y) {
  const double L1 = x[0], a1 = x[1], b1 = x[2];
  const double L2 = y[0], a2 = y[1], b2 = y[2];
  const double Cm = 0.5 * (hypot(a1, b1) + hypot(a2, b2));
  const double Cm7 = pow(Cm, 7.0);
  const double G = 0.5 * (1.0 - sqrt(Cm7 / (Cm7 + pow(25.0, 7.0))));
  const double ap1 = (1.0 + G) * a1, ap2 = (1.0 + G) * a2;
  const double Cp1 = hypot(ap1, b1), Cp2 = hypot(ap2, b2);
  auto hue = [](double b, double ap, double cp) {
    if (cp == 0.0) return 0.0;
    double h = atan2(b, ap) * (180.0 / kPi);
    return h < 0.0 ? h + 360.0 : h;
  };
  const double hp1 = hue(b1, ap1, Cp1), hp2 = hue(b2, ap2, Cp2);
  const bool achromatic = Cp1 * Cp2 == 0.0;
  double dh = hp2 - hp1;
  if (dh > 180.0) dh -= 360.0;
  else if (dh < -180.0) dh += 360.0;
  if (achromatic) dh = 0.0;
  const double dL = L2 - L1, dC = Cp2 - Cp1;
  const double dH = 2.0 * sqrt(Cp1 * Cp2) * sin(rad(dh) / 2.0);
  const double Lm = 0.5 * (L1 + L2), Cpm = 0.5 * (Cp1 + Cp2);
  double hm;
  if (achromatic) hm = hp1 + hp2;
  else if (fabs(hp1 - hp2) <= 180.0) hm = 0.5 * (hp1 + hp2);
  else if (hp1 + hp2 < 360.0) hm = 0.5 * (hp1 + hp2 + 360.0);
  else hm = 0.5 * (hp1 + hp2 - 360.0);
  const double T = 1.0 - 0.17 * cos(rad(hm - 30.0)) + 0.24 * cos(rad(2.0 * hm)) +
                   0.32 * cos(rad(3.0 * hm + 6.0)) - 0.20 * cos(rad(4.0 * hm - 63.0));
  const double dtheta = 30.0 * exp(-((hm - 275.0) / 25.0) * ((hm - 275.0) / 25.0));
  const double Cpm7 = pow(Cpm, 7.0);
  const double RC = 2.0 * sqrt(Cpm7 / (Cpm7 + pow(25.0, 7.0)));
  const double SL = 1.0 + 0.015 * (Lm - 50.0) * (Lm - 50.0) / sqrt(20.0 + (Lm - 50.0) * (Lm - 50.0));
  const double SC = 1.0 + 0.045 * Cpm;
  const double SH = 1.0 + 0.015 * Cpm * T;
  const double RT = -sin(rad(2.0 * dtheta)) * RC;
  const double tl = dL / SL, tc = dC / SC, th = dH / SH;
  return sqrt(tl * tl + tc * tc + th * th + RT * tc * th);
}

double log_binom_tail(int64_t u, int64_t n, double p) {
  const double lp = log(p), lq = log1p(-p);
  const double lgn = lgamma((double)n + 1.0);
  double mx = -INFINITY;
  for (int64_t i = 0; i <= u; ++i) {
    const double t = lgn - lgamma((double)i + 1.0) - lgamma((double)(n - i) + 1.0) + i * lp + (n - i) * lq;
    mx = fmax(mx, t);
  }
  double s = 0.0;
  for (int64_t i = 0; i <= u; ++i) {
    const double t = lgn - lgamma((double)i + 1.0) - lgamma((double)(n - i) + 1.0) + i * lp + (n - i) * lq;
    s += exp(t - mx);
  }
  return mx + log(s);
}

}  // namespace carnator

