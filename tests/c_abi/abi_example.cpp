// A consumer of the C ABI with no Python and no PyTorch: HIP runtime calls
// for memory and streams, and the library's fit, forward and backward.
// Runs one bf16 GELU 3-bit case on the null stream and one fp32 Sigmoid
// 4-bit symmetric case on a created stream, each on a ragged element count,
// and writes the inputs, the table and every output as raw little-endian
// files into the directory given as argv[1]; tests/test_gpu_c_abi.py checks
// them against the CPU oracle.  Exit status 0 when every call succeeded.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "fewbit.h"

namespace {

#define HIP_OK(call)                                                         \
  do {                                                                       \
    hipError_t e_ = (call);                                                  \
    if (e_ != hipSuccess) {                                                  \
      std::fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));        \
      return 1;                                                              \
    }                                                                        \
  } while (0)

// deterministic inputs (64-bit LCG, Knuth's constants), centred uniform
struct Lcg {
  uint64_t s;
  double next() {
    s = s * 6364136223846793005ull + 1442695040888963407ull;
    return static_cast<double>(s >> 11) * (1.0 / 9007199254740992.0) - 0.5;
  }
};

uint16_t to_bf16(float f) {   // round to nearest even, NaN kept quiet
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

bool write_file(const std::string& path, const void* p, size_t bytes) {
  FILE* f = std::fopen(path.c_str(), "wb");
  if (!f) return false;
  const bool ok = std::fwrite(p, 1, bytes, f) == bytes;
  return std::fclose(f) == 0 && ok;
}

int run_case(const char* dir, const char* name, int32_t act, int32_t dtype, int32_t bits,
             int32_t flags, const fewbit_weight& w, int64_t n, double scale, hipStream_t stream,
             int32_t kernel_flags = 0) {
  fewbit_table t;
  int rc = fewbit_fit_table(act, bits, &w, 2000, flags, &t);
  if (rc != FEWBIT_OK) {
    std::fprintf(stderr, "%s: fit: %s\n", name, fewbit_strerror(rc));
    return 1;
  }
  t.flags |= kernel_flags;     // the forward kernel choice, if any
  const size_t esz = dtype == FEWBIT_F32 ? 4 : 2;
  std::vector<uint8_t> x(n * esz), g(n * esz);
  Lcg r{static_cast<uint64_t>(n) * 2654435761u + static_cast<uint64_t>(act)};
  for (int64_t i = 0; i < n; ++i) {
    const float xv = static_cast<float>(r.next() * 2.0 * scale), gv = static_cast<float>(r.next());
    if (dtype == FEWBIT_F32) {
      std::memcpy(&x[i * 4], &xv, 4);
      std::memcpy(&g[i * 4], &gv, 4);
    } else {
      const uint16_t xb = to_bf16(xv), gb = to_bf16(gv);
      std::memcpy(&x[i * 2], &xb, 2);
      std::memcpy(&g[i * 2], &gb, 2);
    }
  }
  const int64_t nw = fewbit_packed_words(n, bits);
  void *dx, *dy, *dg, *dgi;
  uint32_t* dc;
  HIP_OK(hipMalloc(&dx, n * esz));
  HIP_OK(hipMalloc(&dy, n * esz));
  HIP_OK(hipMalloc(&dg, n * esz));
  HIP_OK(hipMalloc(&dgi, n * esz));
  HIP_OK(hipMalloc(reinterpret_cast<void**>(&dc), nw * 4));
  HIP_OK(hipMemcpy(dx, x.data(), n * esz, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dg, g.data(), n * esz, hipMemcpyHostToDevice));
  rc = fewbit_fwd(&t, dtype, dx, dy, dc, n, stream);
  if (rc == FEWBIT_OK) rc = fewbit_bwd(&t, dtype, dg, dc, dgi, n, stream);
  if (rc != FEWBIT_OK) {
    std::fprintf(stderr, "%s: %s\n", name, fewbit_strerror(rc));
    return 1;
  }
  HIP_OK(stream ? hipStreamSynchronize(stream) : hipDeviceSynchronize());
  std::vector<uint8_t> y(n * esz), gi(n * esz), c(nw * 4);
  HIP_OK(hipMemcpy(y.data(), dy, n * esz, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(gi.data(), dgi, n * esz, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(c.data(), dc, nw * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipFree(dx));
  HIP_OK(hipFree(dy));
  HIP_OK(hipFree(dg));
  HIP_OK(hipFree(dgi));
  HIP_OK(hipFree(dc));
  const std::string base = std::string(dir) + "/" + name;
  const bool ok = write_file(base + ".table", &t, sizeof t) && write_file(base + ".x", x.data(), x.size()) &&
                  write_file(base + ".g", g.data(), g.size()) && write_file(base + ".y", y.data(), y.size()) &&
                  write_file(base + ".codes", c.data(), c.size()) &&
                  write_file(base + ".gin", gi.data(), gi.size());
  if (!ok) {
    std::fprintf(stderr, "%s: cannot write outputs\n", name);
    return 1;
  }
  std::printf("%s: n=%lld bits=%d ok\n", name, static_cast<long long>(n), bits);
  return 0;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 2) {
    std::fprintf(stderr, "usage: %s <output directory>\n", argv[0]);
    return 2;
  }
  const fewbit_weight normal{FEWBIT_W_NORMAL, 0, -10.0, 10.0, 0.0, 1.0, 0.0, 1.0};
  const fewbit_weight uniform{FEWBIT_W_UNIFORM, 0, -8.0, 8.0, 0.0, 1.0, 0.0, 1.0};
  // bf16 through the table kernel (chosen in the table), on the null stream
  if (fewbit_fwd16_table_min(FEWBIT_GELU, 3, FEWBIT_BF16) <= 0) return 1;
  if (run_case(argv[1], "gelu_bf16_b3", FEWBIT_GELU, FEWBIT_BF16, 3, 0, normal,
               (int64_t{1} << 22) + 1237, 3.0, nullptr, FEWBIT_FLAG_TABLE_FWD))
    return 1;
  hipStream_t s;
  HIP_OK(hipStreamCreate(&s));
  if (run_case(argv[1], "sigmoid_f32_b4_sym", FEWBIT_SIGMOID, FEWBIT_F32, 4, FEWBIT_FLAG_SYMMETRIC,
               uniform, 1000003, 8.0, s))
    return 1;
  HIP_OK(hipStreamDestroy(s));
  return 0;
}
