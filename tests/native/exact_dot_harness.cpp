// Host build of the library's exact fallback (exact_dot.h) for the CPU tests.
#include <stdint.h>

#include "exact_dot.h"

extern "C" float exact_dot_q22_host(const float* x, const int32_t* tq, int n) {
  return aatc::exact_dot_q22([&](int j) { return x[j]; }, [&](int j) { return tq[j]; }, n);
}
