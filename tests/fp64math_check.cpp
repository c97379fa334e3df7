// Host build of the device fp64 math (paper_2206_00470_amd/csrc/fp64math.hpp)
// checked against the C library: prints the worst error in units in the
// last place of each function over random arguments in its range.
#define ADAPM_HD
#include <cmath>
#include <cstdio>
#include <random>

#include "fp64math.hpp"

static double ulps(double a, double b) {
  if (a == b) return 0.0;
  const double m = std::fabs(b) > 0 ? std::fabs(b) : 1e-300;
  return std::fabs(a - b) / (std::nextafter(m, INFINITY) - m);
}

int main(int argc, char** argv) {
  const long n = argc > 1 ? std::atol(argv[1]) : 2000000;
  std::mt19937_64 g(12345);
  auto unit = [&] { return std::ldexp((double)(g() >> 11), -53); };
  double we = 0, wl = 0, ws = 0, wp = 0;
  for (long i = 0; i < n; ++i) {
    const int kind = (int)(i % 4);
    // exp of t <= 0: wide, moderate, tiny and binade-spread arguments
    double t = kind == 0 ? -800.0 * unit() : kind == 1 ? -40.0 * unit() : kind == 2 ? -1e-3 * unit()
                                                                        : -std::ldexp(unit(), -(int)(g() % 1000));
    const double er = std::exp(t);
    if (er > 1e-300) we = std::fmax(we, ulps(adapm::exp_nonpos(t), er));
    // log(1 + e) for e in [0, 1]
    double e = kind == 3 ? std::ldexp(unit(), -(int)(g() % 1000)) : unit();
    wl = std::fmax(wl, ulps(adapm::log1p_unit(e), std::log1p(e)));
    // sigmoid and softplus over both signs
    const double x = (kind % 2 ? -1.0 : 1.0) * (kind < 2 ? 60.0 : 8.0) * unit();
    double sg, sp;
    adapm::sigmoid_softplus(x, &sg, &sp);
    const double sgr = x >= 0 ? 1.0 / (1.0 + std::exp(-x)) : std::exp(x) / (1.0 + std::exp(x));
    const double spr = x > 0 ? x + std::log1p(std::exp(-x)) : std::log1p(std::exp(x));
    ws = std::fmax(ws, ulps(sg, sgr));
    wp = std::fmax(wp, ulps(sp, spr));
  }
  double s0, p0;
  adapm::sigmoid_softplus(0.0, &s0, &p0);
  std::printf("exp %.2f log1p %.2f sigmoid %.2f softplus %.2f\n", we, wl, ws, wp);
  std::printf("special %.17g %.17g %.17g %.17g %.17g\n", adapm::exp_nonpos(0.0), adapm::exp_nonpos(-746.0),
              adapm::log1p_unit(0.0), s0, p0);
  return 0;
}
