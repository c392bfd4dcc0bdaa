// Host-side library fit (fewbit_fit_table, fewbit_packed_words) under
// AddressSanitizer and UndefinedBehaviorSanitizer: every activation, bit
// width, weight kind and flag, edge grid sizes, and the rejected arguments.
// Built and run on the CPU by tests/test_host_sanitizers.py.  Exit status 0
// when every call returned what it should.
#include <cmath>
#include <cstdio>
#include <initializer_list>

#include "fewbit.h"

static int failures = 0;
#define EXPECT(cond)                                                        \
  do {                                                                      \
    if (!(cond)) {                                                          \
      std::fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                           \
    }                                                                       \
  } while (0)

int main() {
  const fewbit_weight uniform{FEWBIT_W_UNIFORM, 0, -8.0, 8.0, 0.0, 1.0, 0.0, 1.0};
  const fewbit_weight normal{FEWBIT_W_NORMAL, 0, -10.0, 10.0, 0.0, 1.0, 0.0, 1.0};
  const fewbit_weight mixture{FEWBIT_W_MIXTURE, 0, -40.0, 40.0, 0.0, 1.0, 0.01, 10.0};
  const fewbit_weight* weights[] = {&uniform, &normal, &mixture};
  for (int act = FEWBIT_GELU; act <= FEWBIT_SOFTPLUS; ++act)
    for (int bits = 1; bits <= 4; ++bits)
      for (const fewbit_weight* w : weights)
        for (int flags : {0, FEWBIT_FLAG_SYMMETRIC, FEWBIT_FLAG_REFINE}) {
          // the symmetric fit is for even f' (Sigmoid, Tanh)
          if ((flags & FEWBIT_FLAG_SYMMETRIC) && act != FEWBIT_SIGMOID && act != FEWBIT_TANH) continue;
          for (long n_grid : {1L << bits, 301L}) {
            fewbit_table t{};
            const int rc = fewbit_fit_table(act, bits, w, n_grid, flags, &t);
            // ReLU's 1-bit fit is exact; a grid of 2^bits cells may make
            // fp32 boundaries collide (E_NUMERIC); anything else must fit
            EXPECT(rc == FEWBIT_OK || rc == FEWBIT_E_NUMERIC);
            if (rc == FEWBIT_OK) {
              const int K = 1 << bits;
              for (int m = 0; m + 1 < K - 1; ++m) EXPECT(t.s[m] < t.s[m + 1]);
              for (int m = 0; m < K; ++m) EXPECT(std::isfinite(t.v[m]));
              EXPECT(std::isfinite(t.loss) && t.loss >= 0.0);
            }
          }
        }
  fewbit_table t{};
  EXPECT(fewbit_fit_table(FEWBIT_GELU, 0, &normal, 100, 0, &t) == FEWBIT_E_BITS);
  EXPECT(fewbit_fit_table(FEWBIT_GELU, 5, &normal, 100, 0, &t) == FEWBIT_E_BITS);
  EXPECT(fewbit_fit_table(99, 3, &normal, 100, 0, &t) == FEWBIT_E_INVALID);
  EXPECT(fewbit_fit_table(FEWBIT_GELU, 3, nullptr, 100, 0, &t) == FEWBIT_E_NULL);
  EXPECT(fewbit_fit_table(FEWBIT_GELU, 3, &normal, 100, 0, nullptr) == FEWBIT_E_NULL);
  EXPECT(fewbit_fit_table(FEWBIT_GELU, 3, &normal, 7, 0, &t) == FEWBIT_E_INVALID);
  EXPECT(fewbit_fit_table(FEWBIT_GELU, 3, &normal, -1, 0, &t) == FEWBIT_E_INVALID);
  EXPECT(fewbit_fit_table(FEWBIT_GELU, 3, &normal, 100, 64, &t) == FEWBIT_E_INVALID);
  const fewbit_weight bad{FEWBIT_W_NORMAL, 0, 1.0, -1.0, 0.0, 1.0, 0.0, 1.0};
  EXPECT(fewbit_fit_table(FEWBIT_GELU, 3, &bad, 100, 0, &t) == FEWBIT_E_INVALID);
  const fewbit_weight nan_sigma{FEWBIT_W_NORMAL, 0, -1.0, 1.0, 0.0, NAN, 0.0, 1.0};
  EXPECT(fewbit_fit_table(FEWBIT_GELU, 3, &nan_sigma, 100, 0, &t) == FEWBIT_E_INVALID);
  for (int bits = 1; bits <= 4; ++bits)
    for (long n : {0L, 1L, 31L, 32L, 33L, 67108863L, 268435456L})
      EXPECT(fewbit_packed_words(n, bits) == (n * bits + 31) / 32);
  EXPECT(fewbit_packed_words(-1, 3) == -1);
  EXPECT(fewbit_packed_words(10, 0) == -1);
  std::printf("fit driver: %d failure(s)\n", failures);
  return failures == 0 ? 0 : 1;
}
