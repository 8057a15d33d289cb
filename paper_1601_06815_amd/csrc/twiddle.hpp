// Compile-time FFT twiddle factors: cos(2*pi*k/L) and sin(2*pi*k/L), evaluated
// in double precision from their Taylor series after an exact octant
// reduction of the integer angle k/L, then rounded once to float.
//
// Plain C++17 with no HIP dependency, so the host test suite can compile it
// with g++ and compare every entry against the C library's cos/sin.
#pragma once

namespace oaa {
namespace tw {

constexpr double kHalfPi = 1.57079632679489661923132169163975144;

// Taylor series, accurate to a few ulp of double for |x| <= pi/4.
constexpr double sin_series(double x) {
  double term = x, sum = x;
  for (int k = 1; k < 14; ++k) {
    term *= -x * x / double((2 * k) * (2 * k + 1));
    sum += term;
  }
  return sum;
}

constexpr double cos_series(double x) {
  double term = 1.0, sum = 1.0;
  for (int k = 1; k < 14; ++k) {
    term *= -x * x / double((2 * k - 1) * (2 * k));
    sum += term;
  }
  return sum;
}

struct CosSin {
  double c, s;
};

// (cos, sin) of 2*pi*k/L for any integer k and L >= 1.
constexpr CosSin cossin_2pi(long k, long L) {
  long m = k % L;
  if (m < 0) m += L;
  // 2*pi*m/L = q*(pi/2) + phi, phi = (pi/2) * rem / L with rem in [0, L)
  const long q = (4 * m) / L;
  const long rem = 4 * m - q * L;
  double cphi = 0.0, sphi = 0.0;
  if (2 * rem <= L) {
    const double phi = kHalfPi * double(rem) / double(L);
    cphi = cos_series(phi);
    sphi = sin_series(phi);
  } else {  // phi > pi/4: use the complementary angle
    const double psi = kHalfPi * double(L - rem) / double(L);
    cphi = sin_series(psi);
    sphi = cos_series(psi);
  }
  switch (q) {
    case 0: return {cphi, sphi};
    case 1: return {-sphi, cphi};
    case 2: return {-cphi, -sphi};
    default: return {sphi, -cphi};
  }
}

template <int L>
struct Table {
  float c[L];
  float s[L];
  constexpr Table() : c(), s() {
    for (int k = 0; k < L; ++k) {
      const CosSin cs = cossin_2pi(k, L);
      c[k] = float(cs.c);
      s[k] = float(cs.s);
    }
  }
};

template <int L>
inline constexpr Table<L> kTable{};

}  // namespace tw
}  // namespace oaa
