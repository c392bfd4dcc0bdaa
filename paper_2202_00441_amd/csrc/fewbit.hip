// fewbit.hip -- gfx950 kernels and C ABI of the few-bit activation path.
//
// Forward (Listing 1, forward; Eq. (2)): y = f(x) plus, for every element,
// the index of the interval of the piecewise-constant approximation of f'
// it falls in, packed densely at `bits` bits per element.
// Backward (Eq. (1) with f' replaced by the approximation; Listing 1,
// backward): grad_in = grad_out * v[idx].
//
// Both passes are pointwise and bound by HBM bandwidth.  Work is cut into
// wave tiles of 512 consecutive elements, whose codes are exactly 16*b whole
// words, and every 16-byte access instruction of a wave covers 1 KiB of
// contiguous memory.  fp16 / bf16: each lane owns 8 consecutive elements
// (one 16-byte access); their 8 codes make a b-byte field, and the fields
// of 4 neighbouring lanes (one DPP quad) always cover whole words, so lanes
// combine fields with quad permutes instead of atomics or shared memory.
// fp32: a tile is two halves of 256 and each lane owns 4 consecutive
// elements of each half (one 16-byte access per half); the words are then
// gathered from 4b-bit lane fields by cross-lane reads (see fp32 tiles).
// Each packed word has one value, written by its lane (and by lanes that
// store an identical copy, so that full tiles need no masking).
//
// Streams are read and written with non-temporal 16-byte buffer accesses
// (nothing is reused).  Most kernels run one wave per tile (the per-element
// fp16 / bf16 forward one wave per two tiles) and let the hardware
// dispatcher balance the compute units; the table-based fp16 / bf16 forward
// is persistent (see the launch-shape knobs below).
//
// fp16 / bf16 forward.  Output pattern and interval index are functions of
// the 16-bit input pattern alone, so from a size that depends on the type,
// activation and bit width (kTableMinLog2) each workgroup looks both up in
// LDS tables over all 65536 patterns, which it builds itself: the outputs
// (mostly by rule, f where no rule holds) and the indices (4 bits per
// pattern, from the boundaries).  A lookup costs two LDS reads instead of an
// evaluation of f and the compares.  Smaller fp16 / bf16 forwards (and those
// whose f and compares are cheap enough), and every fp32 forward, evaluate f
// and search the boundaries per element.
//
// The fitted table travels as kernel arguments (scalar registers); the
// backward spreads the values over the lanes of one register and reads
// them with cross-lane permutes.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>

#include "../../include/fewbit.h"
#include "fwd16_rules.h"

// Launch-shape knobs (compile time): threads per workgroup, workgroups per
// CU and tiles per wave and loop trip, per kernel.  A positive WG_PER_CU
// caps the grid at that many workgroups per compute unit, and waves then walk
// the tiles (persistent); 0 launches one wave per tile group, and the
// hardware dispatcher hands out workgroups as earlier ones finish.  The
// dispatcher balances the load between compute units, whose streaming rates
// differ by a few per cent from one to another; a persistent grid ends only
// when its slowest unit has walked its share.  The fp16 / bf16 forward holds
// 160 KiB of tables per workgroup (all of a CU's LDS), built at its start, so
// it is persistent with one workgroup per CU.
#ifndef FEWBIT_FWD16_THREADS
#define FEWBIT_FWD16_THREADS 512
#endif
#ifndef FEWBIT_FWD16_WG_PER_CU
#define FEWBIT_FWD16_WG_PER_CU 1
#endif
#ifndef FEWBIT_FWD16_UNROLL
#define FEWBIT_FWD16_UNROLL 4
#endif
// the fp16 / bf16 forward by evaluation (no tables): threads per workgroup,
// and tiles per wave loaded together before they are evaluated
#ifndef FEWBIT_FWD16V_THREADS
#define FEWBIT_FWD16V_THREADS 64
#endif
#ifndef FEWBIT_FWD16V_UNROLL
#define FEWBIT_FWD16V_UNROLL 2
#endif
#ifndef FEWBIT_FWD32_THREADS
#define FEWBIT_FWD32_THREADS 256
#endif
#ifndef FEWBIT_FWD32_WG_PER_CU
#define FEWBIT_FWD32_WG_PER_CU 0
#endif
#ifndef FEWBIT_FWD32_UNROLL
#define FEWBIT_FWD32_UNROLL 1
#endif
#ifndef FEWBIT_BWD32_THREADS
#define FEWBIT_BWD32_THREADS 256
#endif
#ifndef FEWBIT_BWD32_UNROLL
#define FEWBIT_BWD32_UNROLL 1
#endif
#ifndef FEWBIT_NT_LOADS
#define FEWBIT_NT_LOADS 1             // non-temporal stream loads
#endif
#ifndef FEWBIT_NT_STORES
#define FEWBIT_NT_STORES 1            // non-temporal stream stores
#endif

namespace {

constexpr int kWave = 64;
constexpr int kPerLane = 8;                 // elements per lane per 16-bit tile
constexpr int kTile = kWave * kPerLane;     // 512 elements per wave tile
constexpr uint32_t kLaneBytes = 16;         // one 16-byte access per lane and instruction
constexpr uint32_t kSpanBytes = kWave * kLaneBytes;   // 1 KiB per wave instruction

struct TableArgs {
  float s[15];
  float v[16];
};

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Stream accesses go through buffer instructions on a wave-uniform span: a
// resource descriptor for `bytes` bytes from a wave-uniform address (scalar
// registers), plus a per-lane byte offset.  The cache policy is explicit in
// every instruction (the non-temporal hint of plain loads and stores can be
// dropped by the compiler when it merges or moves them), and the hardware
// range check turns any access at or past `bytes` into a zero load or a
// dropped store.  Cache-policy bits: 2 = nt (streaming, not kept in cache).
constexpr int kLoadPolicy = FEWBIT_NT_LOADS ? 2 : 0;
constexpr int kStorePolicy = FEWBIT_NT_STORES ? 2 : 0;

struct Span {
  __amdgpu_buffer_rsrc_t r;
  // 0x00020000: raw (unformatted) 32-bit buffer accesses on gfx9
  __device__ Span(const void* base, uint32_t bytes)
      : r(__builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), 0x00020000)) {}
  __device__ u32x4_t ld16(uint32_t off) const {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kLoadPolicy);
  }
  __device__ void st16(uint32_t off, u32x4_t v) const {
    __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, kStorePolicy);
  }
  __device__ uint32_t ld4(uint32_t off) const {
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kLoadPolicy);
  }
  __device__ void st4(uint32_t off, uint32_t v) const {
    __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, kStorePolicy);
  }
};

// ---------------------------------------------------------------- storage
// Half types: two elements per 32-bit word, element 2k in the low half.
template <int DT>
struct Half;

template <>
struct Half<FEWBIT_BF16> {
  // bfloat16 is the upper half of a binary32: widening is a shift
  __device__ static float lo(uint32_t u) { return __uint_as_float(u << 16); }
  __device__ static float hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }
  __device__ static float widen(uint32_t bits16) { return __uint_as_float(bits16 << 16); }
  // round to nearest even (v_cvt_pk_bf16_f32)
  __device__ static uint32_t pack(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
  }
  // magnitudes from here up: exponent all ones (infinity, NaNs)
  static constexpr uint32_t kSpecialFrom = 0x7F80u;
};

template <>
struct Half<FEWBIT_F16> {
  __device__ static float lo(uint32_t u) {
    return static_cast<float>(__builtin_bit_cast(f16x2_t, u).x);
  }
  __device__ static float hi(uint32_t u) {
    return static_cast<float>(__builtin_bit_cast(f16x2_t, u).y);
  }
  __device__ static float widen(uint32_t bits16) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(bits16)));
  }
  // Round to nearest even from the fp32 value.  The operands pass an empty
  // register barrier first: without it the compiler may fuse the multiply
  // or FMA that produced them into one mixed-precision FMA rounded straight
  // to fp16, which rounds once instead of twice and turns -0 into +0.
  __device__ static uint32_t pack(float a, float b) {
    asm("" : "+v"(a), "+v"(b));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, f16x2_t));
  }
  static constexpr uint32_t kSpecialFrom = 0x7C00u;
};

// element-wise access to 16-bit data for the partial tile at the end
template <int DT>
struct Scalar {
  __device__ static float load(const void* p, int64_t e) {
    return Half<DT>::widen(static_cast<const uint16_t*>(p)[e]);
  }
  __device__ static void store(void* p, int64_t e, float v) {
    static_cast<uint16_t*>(p)[e] = static_cast<uint16_t>(Half<DT>::pack(v, 0.0f) & 0xFFFFu);
  }
};

// ---------------------------------------------------------------- activations
// f evaluated in fp32 with hardware exp2 / reciprocal.  x*Phi(x) and
// x*sigmoid(x) are formed as relu(x) - |x| * tail(|x|), tail the upper tail
// probability, which keeps full relative accuracy on the negative side down
// to the subnormals.
//
// The hardware exponential returns no subnormals (results below 2^-126 come
// back as 0), so each exponential is taken of an argument raised by S and
// the factor 2^S is taken back out of the partner operand of the final
// product, which costs nothing: for GELU out of the reciprocal (its
// constants carry 2^S), for SiLU and sigmoid out of the denominator.  S is
// the smallest shift that keeps every product representable in the output
// type (fp16 outputs underflow long before 2^-126, so S = 0 there).
//
// In the product |x| * tail, |x| is clamped to the largest finite float:
// for x = +-inf the other factor is exactly 0 and the product is 0 (not
// inf * 0), so f(x) = relu(x) without a separate branch; NaN still reaches
// the result through the exponential's argument, which is not clamped.
__device__ inline float finite_abs(float x) { return fminf(fabsf(x), 3.4028234663852886e38f); }

// max(x, -0) as one integer op: the unsigned minimum with the bits of -0
// keeps every float with the sign bit clear (+inf, NaN included) and maps
// every negative input to -0.
__device__ inline float relu(float x) {
  return __uint_as_float(min(__float_as_uint(x), 0x80000000u));
}

// 2^e for -1022 <= e <= 1023, from the exponent field
constexpr double pow2(int e) {
  return __builtin_bit_cast(double, static_cast<uint64_t>(1023 + e) << 52);
}

template <int N>
struct Coefs {
  float c[N];
};

// GELU: the normal upper tail Q(t) = P(Z > t) = r exp2(c(r) - t^2/(2 ln 2))
// with r = 1/(1 + p t) and c a polynomial in r (the form of the Chebyshev
// fitted erfc of Numerical Recipes, coefficients fitted here for a minimal
// maximum relative error on t in [0, 15]):
//   degree 3: max rel. error 1.9e-4  (bf16 results: within 1 ulp)
//   degree 4: max rel. error 5.5e-5  (fp16 results: within 1 ulp)
//   degree 6: max rel. error 1.3e-6  (fp32 results: within 1e-5 rel / 2e-6 abs)
template <int DEG>
struct QFit;
template <>
struct QFit<3> {
  static constexpr float p = 0.36950944455033363f;
  static constexpr float c[4] = {-2.7541667327185095f, 1.3469623570975156f,
                                 0.9101290363759839f, -0.5032013588354882f};
};
template <>
struct QFit<4> {
  static constexpr float p = 0.5063964087913556f;
  static constexpr float c[5] = {-2.3043683184461905f, 1.3894173139728148f,
                                 0.6817571899264395f, -1.149862878045882f,
                                 0.38313433006936115f};
};
template <>
struct QFit<6> {
  static constexpr float p = 0.2715552190762726f;
  static constexpr float c[7] = {-3.204975453658058f, 1.4179583422514952f,
                                 0.7853715466157367f, -0.343943261631901f,
                                 1.2761535905064931f, -1.3184075229241483f,
                                 0.3878445554240053f};
};

// Per output type: GELU polynomial degree and the exponent shifts S.
template <int DT>
struct Prec {                       // fp32
  static constexpr int kGeluDeg = 6, kGeluS = 20, kSiluS = 32, kSigmoidS = 24;
};
template <>
struct Prec<FEWBIT_BF16> {
  static constexpr int kGeluDeg = 3, kGeluS = 16, kSiluS = 16, kSigmoidS = 16;
};
template <>
struct Prec<FEWBIT_F16> {
  static constexpr int kGeluDeg = 4, kGeluS = 0, kSiluS = 0, kSigmoidS = 0;
};

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kHalfLog2e = 0.7213475204444817f;   // 1/(2 ln 2)

template <int DT, int ACT>
struct Act;

template <int DT>
struct Act<DT, FEWBIT_GELU> {
  static constexpr int D = Prec<DT>::kGeluDeg, S = Prec<DT>::kGeluS;
  using F = QFit<D>;
  // coefficients of c in r' = 2^-S r: c_i 2^(S i), and c_0 + S (evaluated
  // at compile time: constant-initialised)
  static constexpr Coefs<D + 1> kCoef = [] {
    Coefs<D + 1> a{};
    for (int i = 0; i <= D; ++i)
      a.c[i] = i == 0 ? F::c[0] + static_cast<float>(S)
                      : static_cast<float>(static_cast<double>(F::c[i]) * pow2(S * i));
    return a;
  }();
  static constexpr float kP = static_cast<float>(F::p * pow2(S));
  static constexpr float kScale = static_cast<float>(pow2(S));
  __device__ static float f(float x) {
    const float t = finite_abs(x);
    const float rs = __builtin_amdgcn_rcpf(fmaf(t, kP, kScale));   // 2^-S r
    float c = kCoef.c[D];
#pragma unroll
    for (int i = D - 1; i >= 0; --i) c = fmaf(c, rs, kCoef.c[i]);
    const float e = __builtin_amdgcn_exp2f(fmaf(x * x, -kHalfLog2e, c));    // 2^S Q(t) / r
    return fmaf(-(t * rs), e, relu(x));   // relu(x) - t Q(t); NaN via x*x
  }
};

template <int DT>
struct Act<DT, FEWBIT_SILU> {
  static constexpr int S = Prec<DT>::kSiluS;
  __device__ static float f(float x) {
    const float e = __builtin_amdgcn_exp2f(fmaf(fabsf(x), -kLog2e, static_cast<float>(S)));  // 2^S e^-t
    constexpr float kScale = static_cast<float>(pow2(S));
    const float r = __builtin_amdgcn_rcpf(e + kScale);  // 1/(2^S (1 + e^-t))
    return fmaf(-(finite_abs(x) * e), r, relu(x));    // relu(x) - t sigma(-t); NaN via e
  }
};

// SiLU, fp16 outputs: x sigma(x) = x / (1 + e^-x) directly.  fp16 outputs
// below 2^-25 round to 0, long before e^-x overflows (x < -88), so the
// negative tail needs neither the split above nor a shift; x is raised to
// -FLT_MAX so that -inf gives -FLT_MAX * 0 = -0 (the limit), and a NaN still
// reaches the result through the exponential.  Six instructions instead of
// eight; every fp16 pattern within one unit in the last place.
template <>
struct Act<FEWBIT_F16, FEWBIT_SILU> {
  __device__ static float f(float x) {
    const float r = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x * -kLog2e));
    return fmaxf(x, -3.4028234663852886e38f) * r;
  }
};

template <int DT>
struct Act<DT, FEWBIT_SIGMOID> {
  static constexpr int S = Prec<DT>::kSigmoidS;
  __device__ static float f(float x) {
    const float t = fabsf(x);
    const float e = __builtin_amdgcn_exp2f(fmaf(t, -kLog2e, static_cast<float>(S)));  // 2^S e^-t
    constexpr float kScale = static_cast<float>(pow2(S));
    const float r = __builtin_amdgcn_rcpf(e + kScale);  // 1/(2^S (1 + e^-t))
    return ((x >= 0.0f) ? kScale : e) * r;   // NaN: e * r is NaN
  }
};

// tanh, every type: 1 - 2 / (e^(2|x|) + 1) with the hardware exponential and
// reciprocal (absolute error about 2^-22, so relative error below 2^-20 where
// |tanh| >= 0.245), and below |x| = 1/4, where that form loses relative
// accuracy, the odd Taylor series to x^9 (first omitted term below 1e-8
// relative), which keeps it down to the subnormals.  The sign is copied from
// x; NaN and infinities follow from the exponential.
template <int DT>
struct Act<DT, FEWBIT_TANH> {
  __device__ static float f(float x) {
    const float t = fabsf(x);
    const float e = __builtin_amdgcn_exp2f(t * (2.0f * kLog2e));
    const float big = fmaf(-2.0f, __builtin_amdgcn_rcpf(e + 1.0f), 1.0f);
    const float z = x * x;
    const float p = fmaf(z, fmaf(z, fmaf(z, fmaf(z, 62.0f / 2835.0f, -17.0f / 315.0f),
                                         2.0f / 15.0f), -1.0f / 3.0f), 1.0f);
    return copysignf(t < 0.25f ? t * p : big, x);
  }
};

template <int DT>
struct Act<DT, FEWBIT_RELU> {
  // +0 for every x <= 0 (-0 included); a NaN fails the compare and is kept
  __device__ static float f(float x) { return x <= 0.0f ? 0.0f : x; }
};

// Klambauer et al. (2017): lambda and lambda * alpha
constexpr float kSeluLambda = 1.0507009873554805f;
constexpr float kSeluLambdaAlpha = 1.7580993408473766f;

// SELU, 16-bit outputs: lambda x, or lambda alpha (e^x - 1) for x <= 0 with
// e^x - 1 taken from the hardware exponential from x = -1/4 down (there
// |e^x - 1| >= 0.22, so its absolute error of ~2^-23 is a relative one below
// 2^-20) and above -1/4 from the Taylor series to x^6 (first omitted term
// below 6e-8 relative), which keeps relative accuracy down to the
// subnormals.  NaN via the exponential; -inf gives -lambda alpha.
template <int DT>
struct Act<DT, FEWBIT_SELU> {
  __device__ static float f(float x) {
    const float e = __builtin_amdgcn_exp2f(x * kLog2e) - 1.0f;
    const float p = x * fmaf(x, fmaf(x, fmaf(x, fmaf(x, fmaf(x, 1.0f / 720.0f, 1.0f / 120.0f), 1.0f / 24.0f),
                                             1.0f / 6.0f), 0.5f), 1.0f);
    const float m = x > -0.25f ? p : e;
    return x > 0.0f ? kSeluLambda * x : kSeluLambdaAlpha * m;
  }
};
template <>
struct Act<FEWBIT_F32, FEWBIT_SELU> {
  // e^x - 1 from the hardware exponential: near 0 the subtraction cancels,
  // so the error is an absolute one of about 2^-23 (times lambda alpha), not
  // a relative one; the fp32 results stay well inside their tolerance (the
  // 16-bit form above adds the series near 0 that fp16 outputs need).  NaN
  // via the exponential, -inf gives -lambda alpha.
  __device__ static float f(float x) {
    const float e = __builtin_amdgcn_exp2f(x * kLog2e);
    return x > 0.0f ? kSeluLambda * x : kSeluLambdaAlpha * (e - 1.0f);
  }
};

// Softplus, 16-bit outputs: max(x, 0) + log(1 + u), u = e^-|x| in (0, 1]: no
// overflow, and relative accuracy in both tails.  log(1 + u) is ln 2 log2(1 + u)
// with the hardware log2 for u >= 2^-5 (rounding 1 + u costs at most 2^-24
// absolute, below 2^-18 relative there) and the series u (1 - u/2 + u^2/3 -
// u^3/4) below (first omitted term below 2^-22 relative).  The exponential is
// taken of an argument raised by S and the series' leading factor keeps the
// 2^S until the end, so bf16 outputs keep their relative accuracy down to
// the subnormals (u far below 2^-126).  NaN via the exponential; +inf gives
// +inf, -inf gives +0.
template <int DT>
struct Act<DT, FEWBIT_SOFTPLUS> {
  static constexpr int S = Prec<DT>::kSigmoidS;
  __device__ static float f(float x) {
    const float es = __builtin_amdgcn_exp2f(fmaf(fabsf(x), -kLog2e, static_cast<float>(S)));  // 2^S u
    constexpr float kUnscale = static_cast<float>(pow2(-S));
    const float u = es * kUnscale;
    const float series = (es * fmaf(u, fmaf(u, fmaf(u, -0.25f, 1.0f / 3.0f), -0.5f), 1.0f)) * kUnscale;
    const float viaLog = __builtin_amdgcn_logf(1.0f + u) * 0.6931471805599453f;
    return relu(x) + (u < 0x1p-5f ? series : viaLog);
  }
};
template <>
struct Act<FEWBIT_F32, FEWBIT_SOFTPLUS> {
  // The same split with hardware exp2 and log2: log(1 + e) = ln 2 log2(1 + e)
  // for e = e^-|x| in (0, 1].  Rounding 1 + e costs at most 2^-24 of
  // absolute error in log2, so the result is within ~2e-7 absolute of the
  // exact value (tiny outputs, x << 0, come back as absolute errors of that
  // size, not relative ones, which the fp32 tolerance allows; the 16-bit
  // form above keeps relative accuracy there).
  __device__ static float f(float x) {
    const float e = __builtin_amdgcn_exp2f(-fabsf(x) * kLog2e);
    return fmaf(__builtin_amdgcn_logf(1.0f + e), 0.6931471805599453f, relu(x));
  }
};

// ---------------------------------------------------------------- classify
// idx = number of boundaries s[m] <= x: half-open intervals [s[m-1], s[m]).
// IEEE compares: NaN gives 0, -0 == +0, subnormals are not flushed.
//
// Branch-free binary search over the sorted boundaries: level L tests the
// boundary s[idx + step - 1] (step = 2^(BITS-1-L)), chosen among the 2^L
// candidates by the answers of the levels before it (a select tree over
// scalar-register values), so BITS compares replace 2^BITS - 1.  A NaN fails
// every test and lands in interval 0, as with the count.
//
// The boundaries are first copied to scalar registers through an empty asm
// barrier: otherwise the compiler turns the selects into indexed loads from
// the kernel-argument block, a memory load per level and element.
struct Bounds {
  float s[15];
};

__device__ inline Bounds bounds_of(const TableArgs& tab) {
  Bounds b;
#pragma unroll
  for (int m = 0; m < 15; ++m) {
    float t = tab.s[m];
    asm("" : "+s"(t));
    b.s[m] = t;
  }
  return b;
}

template <int BITS, int L, int D, int K>
__device__ inline float pick_boundary(const bool (&c)[BITS], const Bounds& bd) {
  if constexpr (D == L) {
    constexpr int step = 1 << (BITS - 1 - L);
    return bd.s[K * 2 * step + step - 1];
  } else {
    return c[D] ? pick_boundary<BITS, L, D + 1, 2 * K + 1>(c, bd)
                : pick_boundary<BITS, L, D + 1, 2 * K>(c, bd);
  }
}

template <int BITS, int L = 0>
__device__ inline void search_levels(float x, const Bounds& bd, bool (&c)[BITS], uint32_t& idx) {
  if constexpr (L < BITS) {
    c[L] = x >= pick_boundary<BITS, L, 0, 0>(c, bd);
    idx += c[L] ? (1u << (BITS - 1 - L)) : 0u;
    search_levels<BITS, L + 1>(x, bd, c, idx);
  }
}

template <int BITS>
__device__ inline uint32_t classify(float x, const Bounds& bd) {
  bool c[BITS] = {};
  uint32_t idx = 0;
  search_levels<BITS>(x, bd, c, idx);
  return idx;
}

// The classification of the per-element kernels and of the code-table
// build.  Up to 3 bits it is the select tree above.  At 4 bits the tree's
// last level alone takes 7 selects, so there the boundaries are spread over
// the lanes of one register (lane i holds s[i], i < 15): the first level
// compares with the middle boundary, held in a scalar register, and each
// later level reads its boundary from the lane the search has reached with
// one cross-lane permute (ds_bpermute), ~3 VALU operations and one permute
// per level.  All 64 lanes must take part in every call (the permutes read
// other lanes).
template <int BITS>
struct Search {
  static constexpr uint32_t K = 1u << BITS;
  static constexpr bool kPermute = BITS == 4;
  Bounds bd;          // the select tree's boundaries (BITS <= 3)
  float mid;          // s[K/2 - 1]
  int lane_bound;     // s[lane] for lane < 15
  uint32_t keep;      // bits of x that are classified: all, or all but the sign
  __device__ Search(const TableArgs& tab, int lane, int symmetric)
      : bd(bounds_of(tab)), keep(symmetric ? 0x7FFFFFFFu : 0xFFFFFFFFu) {
    float v = 0.0f;
#pragma unroll
    for (int m = 0; m < 15; ++m) {
      v = (lane == m) ? bd.s[m] : v;
      if (m == static_cast<int>(K / 2 - 1)) mid = bd.s[m];
    }
    lane_bound = __float_as_int(v);
  }
  // the index of x, or of |x| for a symmetric table (one AND with the mask:
  // -0 becomes +0 and a NaN stays a NaN, as with fabsf)
  __device__ uint32_t code(float x) const { return (*this)(__uint_as_float(__float_as_uint(x) & keep)); }
  // F = F 2^BITS + index of x (or of |x| when SYM), the bits entering one
  // at a time from the most significant: each level's answer is one
  // add-with-carry (F + F + answer), so a lane that shifts in its elements
  // from last to first ends with element j at bits BITS j.  For SYM the
  // absolute value is a source modifier of the compares.
  template <bool SYM>
  __device__ void shift_in(float x, uint32_t& F) const {
    const float v = SYM ? fabsf(x) : x;
    if constexpr (!kPermute) {
      bool c[BITS] = {};
      shift_levels<0>(v, c, F);
    } else {
      F = (F << BITS) | (*this)(v);
    }
  }
  template <int L>
  __device__ void shift_levels(float v, bool (&c)[BITS], uint32_t& F) const {
    if constexpr (L < BITS) {
      c[L] = v >= pick_boundary<BITS, L, 0, 0>(c, bd);
      F = F + F + (c[L] ? 1u : 0u);
      shift_levels<L + 1>(v, c, F);
    }
  }
  __device__ uint32_t operator()(float x) const {
    if constexpr (!kPermute) {
      return classify<BITS>(x, bd);
    } else {
      // a = 4 idx, the byte address ds_bpermute takes; the constant part of
      // each level's address goes into the instruction's offset field
      uint32_t a = x >= mid ? 4u * (K / 2) : 0u;
#pragma unroll
      for (uint32_t step = K / 4; step >= 1; step /= 2) {
        const float b = __int_as_float(
            __builtin_amdgcn_ds_bpermute(static_cast<int>(a + 4u * (step - 1)), lane_bound));
        a += x >= b ? 4u * step : 0u;
      }
      return a >> 2;
    }
  }
};

// ---------------------------------------------------------------- packing
// quad_perm DPP control: lane k of each quad reads lane sel[k] of the quad.
constexpr int quad_perm(int a, int b, int c, int d) { return a | (b << 2) | (c << 4) | (d << 6); }

template <int CTRL>
__device__ inline uint32_t quad_read(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), CTRL, 0xF, 0xF, false));
}

// word i of a code span
__device__ inline void st_word(const Span& c, int i, uint32_t v) { c.st4(static_cast<uint32_t>(i) * 4u, v); }
__device__ inline uint32_t ld_word(const Span& c, int i) { return c.ld4(static_cast<uint32_t>(i) * 4u); }

// Lane field F holds the 8 codes of the lane (8*BITS bits, code j at bit
// BITS*j).  The tile's stream is the lane fields laid end to end, so lane l's
// field starts at stream bit 8*BITS*l.  Writes the words of the tile whose
// index is below `valid` (the rest belong past the end of the buffer).
// Must be called by all 64 lanes together.
template <int BITS>
__device__ inline void pack_store(const Span& out, uint32_t F, int lane, int64_t valid) {
  if constexpr (BITS == 4) {
    if (lane < valid) st_word(out, lane, F);
  } else if constexpr (BITS == 2) {
    const uint32_t nb = quad_read<quad_perm(1, 1, 3, 3)>(F);
    const uint32_t w = F | (nb << 16);
    const int widx = lane >> 1;
    if (!(lane & 1) && widx < valid) st_word(out, widx, w);
  } else if constexpr (BITS == 1) {
    const uint32_t n1 = quad_read<quad_perm(1, 1, 3, 3)>(F);
    const uint32_t a = F | (n1 << 8);
    const uint32_t n2 = quad_read<quad_perm(2, 2, 2, 2)>(a);
    const uint32_t w = a | (n2 << 16);
    const int widx = lane >> 2;
    if (!(lane & 3) && widx < valid) st_word(out, widx, w);
  } else {  // BITS == 3: a quad's 4 x 24 bits are words 3q, 3q+1, 3q+2
    const uint32_t nx = quad_read<quad_perm(1, 2, 3, 3)>(F);
    const int k = lane & 3;
    const uint32_t w = (F >> (8 * k)) | (nx << (24 - 8 * k));
    const int widx = 3 * (lane >> 2) + k;
    if (k < 3 && widx < valid) st_word(out, widx, w);
  }
}

// Inverse of the layout above: the lane's 8*BITS-bit field.  For 1, 2 and 4
// bits a field lies inside one word (lanes that share a word read the same
// address).  For 3 bits lanes 0..2 of each quad read the quad's 3 words with
// one coalesced load; each lane then takes its own word and the one before
// it from the quad and funnel-shifts its 24 bits out.  Must be called by all
// 64 lanes together.
template <int BITS>
__device__ inline uint32_t load_field(const Span& base, int lane, int64_t valid) {
  if constexpr (BITS == 3) {
    const int k = lane & 3;
    const int widx = 3 * (lane >> 2) + k;
    const uint32_t w = (k < 3 && widx < valid) ? ld_word(base, widx) : 0u;
    const uint32_t prev = quad_read<quad_perm(0, 0, 1, 2)>(w);   // word k-1 (k = 0: word 0)
    const uint32_t own = quad_read<quad_perm(0, 1, 2, 2)>(w);    // word k (k = 3: word 2)
    return __builtin_amdgcn_alignbit(own, prev, (24 * k) & 31);
  } else {
    const int widx = (8 * BITS * lane) >> 5;
    const uint32_t v = (widx < valid) ? ld_word(base, widx) : 0u;
    return v >> ((8 * BITS * lane) & 31);
  }
}

// The same two layouts for a full tile, with every lane active: in the
// loops over full tiles no lane is masked off, so no branch splits the loop
// body and the compiler can keep all of a group's loads in flight.  When
// packing, a lane without a word of its own stores an identical copy of a
// neighbour's word to the same address; when unpacking, lane 3 of each quad
// reloads word 2 of the quad, which the permutes never read.
template <int BITS>
__device__ inline void pack_store_full(const Span& out, uint32_t F, int lane) {
  if constexpr (BITS == 4) {
    st_word(out, lane, F);
  } else if constexpr (BITS == 2) {
    const uint32_t lo = quad_read<quad_perm(0, 0, 2, 2)>(F);
    const uint32_t hi = quad_read<quad_perm(1, 1, 3, 3)>(F);
    st_word(out, lane >> 1, lo | (hi << 16));
  } else if constexpr (BITS == 1) {
    const uint32_t a = quad_read<quad_perm(0, 0, 2, 2)>(F) | (quad_read<quad_perm(1, 1, 3, 3)>(F) << 8);
    const uint32_t w = quad_read<quad_perm(0, 0, 0, 0)>(a) | (quad_read<quad_perm(2, 2, 2, 2)>(a) << 16);
    st_word(out, lane >> 2, w);
  } else {  // BITS == 3: lane k of a quad writes word min(k, 2) of the quad
    const int j = min(lane & 3, 2);
    const uint32_t lo = quad_read<quad_perm(0, 1, 2, 2)>(F);
    const uint32_t hi = quad_read<quad_perm(1, 2, 3, 3)>(F);
    st_word(out, 3 * (lane >> 2) + j, (lo >> (8 * j)) | (hi << (24 - 8 * j)));
  }
}

template <int BITS>
__device__ inline uint32_t load_field_full(const Span& base, int lane) {
  if constexpr (BITS == 3) {
    const int k = lane & 3;
    const uint32_t w = ld_word(base, 3 * (lane >> 2) + min(k, 2));
    const uint32_t prev = quad_read<quad_perm(0, 0, 1, 2)>(w);   // word k-1 (k = 0: word 0)
    const uint32_t own = quad_read<quad_perm(0, 1, 2, 2)>(w);    // word k (k = 3: word 2)
    return __builtin_amdgcn_alignbit(own, prev, (24 * k) & 31);
  } else {
    return ld_word(base, (8 * BITS * lane) >> 5) >> ((8 * BITS * lane) & 31);
  }
}

struct WaveIndex {
  int lane;
  int64_t wave, nwaves;
};
// The waves of every workgroup, numbered across the grid.  The waves per
// workgroup come from the launch's THREADS as a compile-time constant:
// blockDim would be a vector load from the dispatch packet, waited for
// before the first stream load.
template <int THREADS>
__device__ inline WaveIndex wave_index() {
  constexpr int kPerBlock = THREADS / kWave;
  // the wave's number within its workgroup is the same in all its lanes;
  // readfirstlane tells the compiler so, which keeps tile addresses scalar
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x / kWave));
  return {static_cast<int>(threadIdx.x & (kWave - 1)),
          static_cast<int64_t>(blockIdx.x) * kPerBlock + w,
          static_cast<int64_t>(gridDim.x) * kPerBlock};
}

// ---------------------------------------------------------------- forward, fp16 / bf16
// For 16-bit inputs both results of the forward are functions of the input
// bit pattern alone, so every workgroup holds two tables over all 65536
// patterns in LDS:
//   ylut  the output pattern of f(x), 128 KiB;
//   clut  the interval index, 4 bits per pattern: byte q holds pattern 2q in
//         its low and pattern 2q+1 in its high nibble, 32 KiB.
// A tile then costs two LDS reads and a few integer operations per element
// instead of an evaluation of f and the compares.
//
// ylut depends only on the activation and the storage type, and most of it
// follows a simple rule (fwd16_rules.h, written by gen_fwd16_rules.py: the
// table is 512 blocks of 128 patterns; runs of blocks are the input itself,
// one constant, RNE(x / 2), RNE(lambda x), or need f).  Every workgroup fills
// its ylut from those runs, which travel as kernel arguments, and evaluates f
// (the fp32 f of the per-element path, then one rounding) only in the blocks
// no rule covers: for bf16 GELU 30 blocks of 512.  clut depends on the
// boundaries and is built by every workgroup: the index is monotone in the
// pattern within one sign, so each thread classifies only the two ends of its
// segment of patterns and fills it if they agree; the few segments that hold
// a boundary, infinities or NaNs are then classified pattern by pattern by the
// whole wave.  Neither table outlives the workgroup: the library keeps no
// device memory.
struct OutRuns {
  uint32_t r[fwd16_rules::kMaxRuns];
};

// ylut from the runs, by each wave on its own (no barrier, no scratch):
//   1. wave w fills the 1 KiB chunks w, w + 8, ... of ylut (lane l the 16
//      bytes at 16 l, so one store instruction covers consecutive banks) in
//      the blocks whose rule is integer work on the patterns: IDENTITY,
//      CONST and HALF (one exponent step down).  The chunks' 64 blocks are
//      the wave's: lane l finds the run of block 4 w + 32 (l / 4) + l mod 4
//      and the lanes of each chunk read it with one cross-lane permute.
//      Branch-free: every lane forms both candidates and stores only in
//      those blocks;
//   2. the blocks of the runs that need arithmetic (EVAL: the kernel's f;
//      SCALE), numbered in order, go to the waves in turn; 2 patterns per
//      lane, the rule uniform over the wave.  The two steps store to
//      different blocks.
template <int DT, int ACT>
__device__ void build_output_table(uint16_t* ylut, const OutRuns& runs) {
  using namespace fwd16_rules;
  static_assert(FEWBIT_FWD16_THREADS == 512, "8 waves, 16 chunks each");
  constexpr uint32_t kWaves = FEWBIT_FWD16_THREADS / kWave;
  constexpr uint32_t kChunks = 128u / kWaves;           // 1 KiB chunks per wave
  // x / 2 as one exponent step down (subtracted from both halves of a word)
  constexpr uint32_t kHalfStep = DT == FEWBIT_BF16 ? 0x00800080u : 0x04000400u;
  using H = Half<DT>;
  uint32_t R[kMaxRuns];
#pragma unroll
  for (int j = 0; j < kMaxRuns; ++j) {
    uint32_t t = runs.r[j];
    asm("" : "+s"(t));         // keep the descriptors in scalar registers
    R[j] = t;
  }
  const uint32_t lane = threadIdx.x & (kWave - 1);
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  uint32_t mine = R[0];
  {
    const uint32_t blk = 4u * wave + 32u * (lane >> 2) + (lane & 3u);
#pragma unroll
    for (int j = 1; j < kMaxRuns; ++j) mine = (R[j] & 1023u) <= blk ? R[j] : mine;
  }
  // all permutes first: each waits in LDS order, so issuing one after the
  // previous chunk's store would wait for that store too
  uint32_t descs[kChunks];
#pragma unroll
  for (uint32_t i = 0; i < kChunks; ++i)
    descs[i] = static_cast<uint32_t>(
        __builtin_amdgcn_ds_bpermute(static_cast<int>(4u * (4u * i + (lane >> 4))), static_cast<int>(mine)));
#pragma unroll
  for (uint32_t i = 0; i < kChunks; ++i) {
    const uint32_t p0 = (wave + kWaves * i) * 512u + lane * 8u;   // the lane's first pattern
    const uint32_t desc = descs[i];
    const uint32_t rule = (desc >> 12) & 15u;
    // word e of the lane's 4: base + e step, the pattern pair (one exponent
    // step down for HALF) or the constant
    const uint32_t pair = (p0 | ((p0 + 1u) << 16)) - (rule == HALF ? kHalfStep : 0u);
    // a bit select through a mask in a register: as a ?: the compiler
    // branches around the constant's multiply
    uint32_t is_const = rule == CONST ? ~0u : 0u;
    asm("" : "+v"(is_const));
    const uint32_t base = (((desc >> 16) * 0x10001u) & is_const) | (pair & ~is_const);
    const uint32_t step = 0x00020002u & ~is_const;
    const u32x4_t v = {base, base + step, base + 2u * step, base + 3u * step};
    if (rule == IDENTITY || rule == CONST || rule == HALF) *reinterpret_cast<u32x4_t*>(ylut + p0) = v;
  }
  // the blocks needing arithmetic, numbered across the runs in order: the
  // k-th goes to wave k mod 8
  uint32_t* ylut32 = reinterpret_cast<uint32_t*>(ylut);
  uint32_t before = 0;          // such blocks in the runs before run j
#pragma unroll
  for (int j = 0; j < kMaxRuns; ++j) {
    const uint32_t rule = (R[j] >> 12) & 15u;
    const uint32_t start = R[j] & 1023u;
    const uint32_t end = j + 1 < kMaxRuns ? min(R[j + 1] & 1023u, 512u) : 512u;
    if (start >= 512u || (rule != EVAL && rule != SCALE)) continue;
    const uint32_t first = start + ((wave + 8u - (before & 7u)) & 7u);
    before += end - start;
    for (uint32_t blk = first; blk < end; blk += 8u) {
      const uint32_t p = blk * 128u + 2u * lane;
      const float x0 = H::widen(p), x1 = H::widen(p + 1u);
      ylut32[blk * 64u + lane] = rule == EVAL ? H::pack(Act<DT, ACT>::f(x0), Act<DT, ACT>::f(x1))
                                              : H::pack(x0 * kSeluLambda, x1 * kSeluLambda);
    }
  }
}

template <int DT, int BITS>
__device__ void build_code_table(uint8_t* clut, const TableArgs& tab, int symmetric) {
  // each thread owns one aligned segment of kSeg patterns (kSeg / 2 bytes)
  constexpr uint32_t kSeg = 65536u / FEWBIT_FWD16_THREADS;
  static_assert(kSeg >= 32 && kSeg <= 32768 && 65536u % FEWBIT_FWD16_THREADS == 0,
                "segments of whole 16-byte stores within one sign");
  // every call below is made by all 64 lanes of the wave, as Search's
  // permutes require: the segment loop takes two patterns per lane and kSeg
  // is a multiple of 128, so all lanes run it equally often
  static_assert(kSeg % (2 * kWave) == 0, "whole waves in the segment loop");
  const Search<BITS> cl(tab, static_cast<int>(threadIdx.x & (kWave - 1)), symmetric);
  auto code_of = [&](uint32_t p) { return cl.code(Half<DT>::widen(p)); };
  const uint32_t p0 = threadIdx.x * kSeg;
  const uint32_t last = p0 + kSeg - 1u;
  // the index is monotone in the pattern within one sign, so a segment
  // whose two ends agree is uniform, unless it reaches the infinities and
  // NaNs at the top of its sign (exponent all ones)
  const bool special = (last & 0x7FFFu) >= Half<DT>::kSpecialFrom;
  const uint32_t a = code_of(p0), b = code_of(last);
  const bool uniform = !special && a == b;
  if (uniform) {
    const uint32_t rep = a * 0x11111111u;
#pragma unroll
    for (uint32_t i = 0; i < kSeg / 32u; ++i)
      reinterpret_cast<u32x4_t*>(clut + p0 / 2u)[i] = (u32x4_t){rep, rep, rep, rep};
  }
  // the other segments are classified pattern by pattern by the whole wave
  const uint32_t lane = threadIdx.x & (kWave - 1), first = threadIdx.x - lane;
  uint64_t todo = __ballot(!uniform);
  while (todo) {
    const uint32_t l = static_cast<uint32_t>(__builtin_ctzll(todo));
    todo &= todo - 1u;
    const uint32_t q0 = (first + l) * kSeg;
    for (uint32_t j = 2u * lane; j < kSeg; j += 2u * kWave)
      clut[(q0 + j) / 2u] = static_cast<uint8_t>(code_of(q0 + j) | (code_of(q0 + j + 1u) << 4));
  }
}

__device__ inline uint32_t code_of_pattern(const uint8_t* clut, uint32_t p) {
  return (static_cast<uint32_t>(clut[p >> 1]) >> ((p & 1u) << 2)) & 15u;
}

template <int BITS>
__device__ inline void fwd16_tile(u32x4_t in, const uint16_t* ylut, const uint8_t* clut,
                                  u32x4_t& out, uint32_t& F) {
  F = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t w = in[k];
    const uint32_t lo = w & 0xFFFFu, hi = w >> 16;
    out[k] = static_cast<uint32_t>(ylut[lo]) | (static_cast<uint32_t>(ylut[hi]) << 16);
    F |= (code_of_pattern(clut, lo) << (2 * k * BITS)) |
         (code_of_pattern(clut, hi) << ((2 * k + 1) * BITS));
  }
}

template <int DT, int BITS, int ACT>
__global__ __launch_bounds__(FEWBIT_FWD16_THREADS) void fwd16_kernel(
    const uint16_t* x, uint16_t* y, uint32_t* __restrict__ codes, int64_t n, int64_t nwords,
    TableArgs tab, int symmetric, OutRuns runs) {
  constexpr int U = FEWBIT_FWD16_UNROLL;
  constexpr int kWords = 16 * BITS;
  // clut first: ylut's 32 KiB offset then fits the LDS instruction's
  // immediate offset field
  __shared__ __attribute__((aligned(16))) uint8_t tables[32768 + 2 * 65536];
  uint8_t* clut = tables;
  uint16_t* ylut = reinterpret_cast<uint16_t*>(tables + 32768);
  const WaveIndex wi = wave_index<FEWBIT_FWD16_THREADS>();
  const int64_t full = n / kTile;
  const int64_t groups = full / U;
  const int64_t lane_off = static_cast<int64_t>(wi.lane) * kPerLane;
  const uint32_t lane_b = static_cast<uint32_t>(wi.lane) * kLaneBytes;

  // the wave's first tile group is loaded before the tables are built, so
  // its memory latency passes during the build
  int64_t gi = wi.wave;
  u32x4_t in[U];
  if (gi < groups) {
#pragma unroll
    for (int u = 0; u < U; ++u) in[u] = Span(x + (gi * U + u) * kTile, kSpanBytes).ld16(lane_b);
  }
  build_output_table<DT, ACT>(ylut, runs);
  build_code_table<DT, BITS>(clut, tab, symmetric);
  __syncthreads();

  for (bool loaded = true; gi < groups; gi += wi.nwaves, loaded = false) {
    const int64_t t0 = gi * U;
    u32x4_t out[U];
    uint32_t F[U];
    if (!loaded) {
#pragma unroll
      for (int u = 0; u < U; ++u) in[u] = Span(x + (t0 + u) * kTile, kSpanBytes).ld16(lane_b);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) fwd16_tile<BITS>(in[u], ylut, clut, out[u], F[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      Span(y + (t0 + u) * kTile, kSpanBytes).st16(lane_b, out[u]);
      pack_store_full<BITS>(Span(codes + (t0 + u) * kWords, kWords * 4), F[u], wi.lane);
    }
  }
  for (int64_t t = groups * U + wi.wave; t < full; t += wi.nwaves) {
    u32x4_t out;
    uint32_t F;
    fwd16_tile<BITS>(Span(x + t * kTile, kSpanBytes).ld16(lane_b), ylut, clut, out, F);
    Span(y + t * kTile, kSpanBytes).st16(lane_b, out);
    pack_store_full<BITS>(Span(codes + t * kWords, kWords * 4), F, wi.lane);
  }
  // the partial tile at the end, if any, goes to the wave that would own it
  if (n % kTile != 0 && wi.wave == full % wi.nwaves) {
    const int64_t t = full;
    uint32_t F = 0;
#pragma unroll
    for (int j = 0; j < kPerLane; ++j) {
      const int64_t e = t * kTile + lane_off + j;
      if (e < n) {
        const uint32_t p = x[e];
        y[e] = ylut[p];
        F |= code_of_pattern(clut, p) << (BITS * j);
      }
    }
    const int64_t wbase = t * kWords;
    pack_store<BITS>(Span(codes + wbase, kWords * 4), F, wi.lane, nwords - wbase);
  }
}

// fp16 / bf16 forward by evaluation: f and the compares for every element,
// no tables.  The table kernel above builds its tables in every workgroup
// and runs a persistent grid; below the sizes of kTableMinLog2 this kernel,
// with no setup and a dispatcher-balanced grid of two-tile waves, is
// faster.  Where the table kernel evaluates f (the blocks no rule covers) it
// uses this same f and rounding.
//
// The full tiles of one wave: y from the fp32 f, and the codes shifted into
// the lane's field from its last element to its first (element j of the
// lane's 8 at bits BITS j).  SYM: the table is symmetric, the index is that
// of |x|.  The wave takes its tiles in groups of U consecutive ones and
// issues all U loads before it evaluates the first, so its next loads are in
// flight while it computes (one tile per wave leaves the memory idle during
// the evaluation, which is long next to the streaming); the whole tiles past
// the last group go one at a time.
template <int DT, int BITS, int ACT, bool SYM>
__device__ inline void fwd16v_tile(u32x4_t in, const Search<BITS>& cl, u32x4_t& out, uint32_t& F) {
  using H = Half<DT>;
  F = 0;
#pragma unroll
  for (int k = 3; k >= 0; --k) {
    const float a = H::lo(in[k]), b = H::hi(in[k]);
    cl.template shift_in<SYM>(b, F);
    cl.template shift_in<SYM>(a, F);
    out[k] = H::pack(Act<DT, ACT>::f(a), Act<DT, ACT>::f(b));
  }
}

template <int DT, int BITS, int ACT, bool SYM>
__device__ inline void fwd16v_tiles(const uint16_t* x, uint16_t* y, uint32_t* codes, int64_t full,
                                    const WaveIndex& wi, const Search<BITS>& cl) {
  constexpr int U = FEWBIT_FWD16V_UNROLL;
  constexpr int kWords = 16 * BITS;
  const uint32_t lane_b = static_cast<uint32_t>(wi.lane) * kLaneBytes;
  const int64_t groups = full / U;
  for (int64_t g = wi.wave; g < groups; g += wi.nwaves) {
    const int64_t t0 = g * U;
    u32x4_t in[U];
#pragma unroll
    for (int u = 0; u < U; ++u) in[u] = Span(x + (t0 + u) * kTile, kSpanBytes).ld16(lane_b);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      u32x4_t out;
      uint32_t F;
      fwd16v_tile<DT, BITS, ACT, SYM>(in[u], cl, out, F);
      Span(y + (t0 + u) * kTile, kSpanBytes).st16(lane_b, out);
      pack_store_full<BITS>(Span(codes + (t0 + u) * kWords, kWords * 4), F, wi.lane);
    }
  }
  for (int64_t t = groups * U + wi.wave; t < full; t += wi.nwaves) {
    u32x4_t out;
    uint32_t F;
    fwd16v_tile<DT, BITS, ACT, SYM>(Span(x + t * kTile, kSpanBytes).ld16(lane_b), cl, out, F);
    Span(y + t * kTile, kSpanBytes).st16(lane_b, out);
    pack_store_full<BITS>(Span(codes + t * kWords, kWords * 4), F, wi.lane);
  }
}

template <int DT, int BITS, int ACT>
__global__ __launch_bounds__(FEWBIT_FWD16V_THREADS) void fwd16v_kernel(
    const uint16_t* x, uint16_t* y, uint32_t* __restrict__ codes, int64_t n, int64_t nwords,
    TableArgs tab, int symmetric) {
  constexpr int kWords = 16 * BITS;
  const WaveIndex wi = wave_index<FEWBIT_FWD16V_THREADS>();
  const Search<BITS> cl(tab, wi.lane, symmetric);
  const int64_t full = n / kTile;
  const int64_t lane_off = static_cast<int64_t>(wi.lane) * kPerLane;
  if (symmetric)
    fwd16v_tiles<DT, BITS, ACT, true>(x, y, codes, full, wi, cl);
  else
    fwd16v_tiles<DT, BITS, ACT, false>(x, y, codes, full, wi, cl);
  // the partial tile at the end, if any, goes to the wave that would own it
  if (n % kTile != 0 && wi.wave == full % wi.nwaves) {
    const int64_t t = full;
    uint32_t F = 0;
#pragma unroll
    for (int j = 0; j < kPerLane; ++j) {
      const int64_t e = t * kTile + lane_off + j;
      const float v = e < n ? Half<DT>::widen(x[e]) : 0.0f;
      const uint32_t c = cl.code(v);                          // all lanes
      if (e < n) {
        y[e] = static_cast<uint16_t>(Half<DT>::pack(Act<DT, ACT>::f(v), 0.0f) & 0xFFFFu);
        F |= c << (BITS * j);
      }
    }
    const int64_t wbase = t * kWords;
    pack_store<BITS>(Span(codes + wbase, kWords * 4), F, wi.lane, nwords - wbase);
  }
}

// ---------------------------------------------------------------- fp32 tiles
// An fp32 tile is 512 elements in two halves of 256; lane l holds elements
// 4l .. 4l+3 of each half, so each 16-byte access instruction covers 1 KiB
// of contiguous memory.  (Eight consecutive elements per lane would need two
// accesses 32 bytes apart per lane, each instruction touching only every
// other 16 bytes of its span, which streams far below the contiguous rate.)
// In stream order a half's codes are then the lanes' fields of 4*BITS bits
// laid end to end, 8*BITS words per half, 16*BITS per tile.
template <int BITS>
struct Codes32 {
  static constexpr int FB = 4 * BITS;                  // field bits per lane and half
  static constexpr uint32_t kMask = (1u << FB) - 1u;
  static constexpr int kHalfWords = 8 * BITS;
  static constexpr int kWords = 16 * BITS;
  // most lanes whose fields meet one word: 32 / FB when fields tile words,
  // else a partial field at each end (for 12-bit fields: 4 lanes)
  static constexpr int kSources = 32 / FB + ((32 % FB) ? 2 : 0);
};

// Every lane builds word q = lane mod 16*BITS of the tile from the fields
// of the lanes it covers (cross-lane reads of f0 | f1 << 16), and stores it;
// lanes past 16*BITS store identical copies.  FULL: the whole tile exists,
// so no store is masked off; else only words below `valid` are stored.
template <int BITS, bool FULL>
__device__ inline void pack_store32(const Span& out, uint32_t f0, uint32_t f1, int lane,
                                    int64_t valid) {
  using C = Codes32<BITS>;
  const uint32_t both = f0 | (f1 << 16);
  const int q = lane % C::kWords;
  const int v = q / C::kHalfWords, w = q % C::kHalfWords;
  const int a = (32 * w) / C::FB, o = (32 * w) % C::FB;
  uint32_t word = 0;
#pragma unroll
  for (int i = 0; i < C::kSources; ++i) {
    const uint32_t f = (static_cast<uint32_t>(__shfl(static_cast<int>(both), (a + i) & 63)) >>
                        (16 * v)) & C::kMask;
    const int sh = i * C::FB - o;                      // bit position of the field in the word
    word |= (i == 0) ? (f >> o) : (sh < 32 ? f << sh : 0u);
  }
  if (FULL || q < valid) st_word(out, q, word);
}

// The field of lane `lane` in half v: the one or two words it spans,
// funnel-shifted.  FULL: every word of the tile exists; else words from
// `valid` on read as 0.
template <int BITS, bool FULL>
__device__ inline uint32_t load_field32(const Span& base, int v, int lane, int64_t valid) {
  using C = Codes32<BITS>;
  const int b0 = lane * C::FB;
  const int i0 = v * C::kHalfWords + (b0 >> 5);
  const int i1 = min(i0 + 1, C::kWords - 1);           // unused unless the field straddles
  const uint32_t lo = (FULL || i0 < valid) ? ld_word(base, i0) : 0u;
  const uint32_t hi = (FULL || i1 < valid) ? ld_word(base, i1) : 0u;
  return __builtin_amdgcn_alignbit(hi, lo, b0 & 31) & C::kMask;
}

// ---------------------------------------------------------------- forward, fp32
template <int BITS, int ACT>
__device__ inline void fwd32_half(u32x4_t in, const Search<BITS>& cl, u32x4_t& out, uint32_t& f) {
  f = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float xv = __uint_as_float(in[j]);
    out[j] = __float_as_uint(Act<FEWBIT_F32, ACT>::f(xv));
    f |= cl.code(xv) << (BITS * j);
  }
}

template <int BITS, int ACT>
__global__ __launch_bounds__(FEWBIT_FWD32_THREADS) void fwd32_kernel(
    const float* x, float* y, uint32_t* __restrict__ codes, int64_t n, int64_t nwords,
    TableArgs tab, int symmetric) {
  constexpr int U = FEWBIT_FWD32_UNROLL;
  constexpr int kWords = Codes32<BITS>::kWords;
  const WaveIndex wi = wave_index<FEWBIT_FWD32_THREADS>();
  const Search<BITS> cl(tab, wi.lane, symmetric);
  const int64_t full = n / kTile;
  const int64_t groups = full / U;
  const int64_t lane_off = static_cast<int64_t>(wi.lane) * 4;
  const uint32_t lane_b = static_cast<uint32_t>(wi.lane) * kLaneBytes;

  for (int64_t gi = wi.wave; gi < groups; gi += wi.nwaves) {
    const int64_t t0 = gi * U;
    u32x4_t in[U][2], out[U][2];
    uint32_t f[U][2];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int h = 0; h < 2; ++h) in[u][h] = Span(x + (t0 + u) * kTile + h * 256, kSpanBytes).ld16(lane_b);
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int h = 0; h < 2; ++h) fwd32_half<BITS, ACT>(in[u][h], cl, out[u][h], f[u][h]);
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int h = 0; h < 2; ++h) Span(y + (t0 + u) * kTile + h * 256, kSpanBytes).st16(lane_b, out[u][h]);
      pack_store32<BITS, true>(Span(codes + (t0 + u) * kWords, kWords * 4), f[u][0], f[u][1], wi.lane, kWords);
    }
  }
  for (int64_t t = groups * U + wi.wave; t < full; t += wi.nwaves) {
    u32x4_t out[2];
    uint32_t f[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      fwd32_half<BITS, ACT>(Span(x + t * kTile + h * 256, kSpanBytes).ld16(lane_b), cl, out[h], f[h]);
      Span(y + t * kTile + h * 256, kSpanBytes).st16(lane_b, out[h]);
    }
    pack_store32<BITS, true>(Span(codes + t * kWords, kWords * 4), f[0], f[1], wi.lane, kWords);
  }
  // the partial tile at the end, if any, goes to the wave that would own it
  if (n % kTile != 0 && wi.wave == full % wi.nwaves) {
    const int64_t t = full;
    uint32_t f[2] = {0u, 0u};
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t e = t * kTile + h * 256 + lane_off + j;
        const float xv = e < n ? x[e] : 0.0f;
        const uint32_t c = cl.code(xv);                     // all lanes
        if (e < n) {
          y[e] = Act<FEWBIT_F32, ACT>::f(xv);
          f[h] |= c << (BITS * j);
        }
      }
    const int64_t wbase = t * kWords;
    pack_store32<BITS, false>(Span(codes + wbase, kWords * 4), f[0], f[1], wi.lane, nwords - wbase);
  }
}

// ---------------------------------------------------------------- backward
// The K values of the table live in one register of each wave, lane i
// holding v[i mod K] (K <= 16 divides 64), and an element's value is read
// from the lane its code names with one cross-lane permute (ds_bpermute).
// No LDS array is filled and no barrier is taken, so a wave issues its
// stream loads as soon as it starts: the backward runs as a grid of
// one-wave workgroups, one tile each, and the hardware dispatcher streams
// them through the device.
template <int BITS>
struct Values {
  int lane_value;
  __device__ explicit Values(const TableArgs& tab) {
    // lane c < K holds v[c] (a chain of selects over scalar registers); the
    // permutes read no other lane.  The values pass an empty asm barrier
    // first, which keeps them in scalar registers: otherwise the compiler
    // may turn the chain into a per-lane load from the kernel-argument
    // block, a vector memory load whose wait would hold back the stream
    // loads.
    const int lane = static_cast<int>(threadIdx.x & (kWave - 1));
    float v = 0.0f;
#pragma unroll
    for (int c = 0; c < (1 << BITS); ++c) {
      float t = tab.v[c];
      asm("" : "+s"(t));
      v = lane == c ? t : v;
    }
    lane_value = __float_as_int(v);
  }
  // v[c] for the code c of this lane; all 64 lanes must take part
  __device__ float operator()(uint32_t c) const {
    return __int_as_float(__builtin_amdgcn_ds_bpermute(static_cast<int>(c << 2), lane_value));
  }
};

template <int DT, int BITS>
__device__ inline u32x4_t grad16_tile(u32x4_t g, uint32_t F, const Values<BITS>& val) {
  using H = Half<DT>;
  constexpr uint32_t kMask = (1u << BITS) - 1u;
  u32x4_t out;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float v0 = val((F >> (2 * k * BITS)) & kMask);
    const float v1 = val((F >> ((2 * k + 1) * BITS)) & kMask);
    out[k] = H::pack(H::lo(g[k]) * v0, H::hi(g[k]) * v1);   // fp32 products, then RNE
  }
  return out;
}

// The 16-bit backward runs one-wave workgroups, one tile each.  At 1 and 3
// bits a tile's code span (64 or 192 bytes) is not a whole number of 128-byte
// lines: tiles 2p and 2p+1 share one line.  Read by waves on different XCDs,
// whose L2 caches are separate, that line would be fetched from memory twice
// (a third of the code stream again at 3 bits).  So workgroup u takes tile
// tile_of_unit(u): within each run of 16 workgroups, workgroups r and r + 8
// take the two tiles of pair r.  The dispatcher hands workgroups to the 8
// XCDs in turn, so the two land on the same XCD, one after the other, and the
// shared line is fetched once.  The grid is a whole number of such runs;
// units whose tile lies past the end do nothing.
template <int BITS>
struct BwdOrder {
  static constexpr bool kPaired = BITS == 1 || BITS == 3;
  static constexpr int64_t kRun = kPaired ? 16 : 1;
  __host__ __device__ static int64_t tile_of_unit(int64_t u) {
    if constexpr (kPaired) {
      const int64_t r = u & 15;
      return (u - r) + 2 * (r & 7) + (r >> 3);
    } else {
      return u;
    }
  }
  // the inverse: the unit that takes tile t
  __host__ __device__ static int64_t unit_of_tile(int64_t t) {
    if constexpr (kPaired) {
      const int64_t q = t & 15;
      return (t - q) + 8 * (q & 1) + (q >> 1);
    } else {
      return t;
    }
  }
};

template <int DT, int BITS>
__device__ inline void bwd16_full_tile(const uint16_t* g, const uint32_t* codes, uint16_t* gin,
                                       int64_t t, int lane, const TableArgs& tab) {
  constexpr int kWords = 16 * BITS;
  const uint32_t lane_b = static_cast<uint32_t>(lane) * kLaneBytes;
  const u32x4_t in = Span(g + t * kTile, kSpanBytes).ld16(lane_b);
  const uint32_t F = load_field_full<BITS>(Span(codes + t * kWords, kWords * 4), lane);
  // the stream loads are in flight before the values are put in place
  __builtin_amdgcn_sched_barrier(0);
  const Values<BITS> val(tab);
  Span(gin + t * kTile, kSpanBytes).st16(lane_b, grad16_tile<DT, BITS>(in, F, val));
}

template <int DT, int BITS>
__global__ __launch_bounds__(kWave) void bwd_kernel(
    const uint16_t* g, const uint32_t* __restrict__ codes, uint16_t* gin, int64_t n,
    int64_t nwords, TableArgs tab) {
  constexpr int kWords = 16 * BITS;
  constexpr uint32_t kMask = (1u << BITS) - 1u;
  constexpr int64_t kRun = BwdOrder<BITS>::kRun;
  const WaveIndex wi = wave_index<kWave>();
  const int64_t full = n / kTile;
  const int64_t units = (full + kRun - 1) / kRun * kRun;

  // one unit per wave unless the grid was capped (see grid_for)
  for (int64_t u = wi.wave; u < units; u += wi.nwaves) {
    const int64_t t = BwdOrder<BITS>::tile_of_unit(u);
    if (t < full) bwd16_full_tile<DT, BITS>(g, codes, gin, t, wi.lane, tab);
  }
  // the partial tile at the end, if any, goes to the wave of its unit
  if (n % kTile != 0 && wi.wave == BwdOrder<BITS>::unit_of_tile(full) % wi.nwaves) {
    const Values<BITS> val(tab);
    const int64_t t = full;
    const int64_t wbase = t * kWords;
    const int64_t lane_off = static_cast<int64_t>(wi.lane) * kPerLane;
    const uint32_t F = load_field<BITS>(Span(codes + wbase, kWords * 4), wi.lane, nwords - wbase);
    float v[kPerLane];
#pragma unroll
    for (int j = 0; j < kPerLane; ++j) v[j] = val((F >> (BITS * j)) & kMask);   // all lanes
#pragma unroll
    for (int j = 0; j < kPerLane; ++j) {
      const int64_t e = t * kTile + lane_off + j;
      if (e < n) Scalar<DT>::store(gin, e, Scalar<DT>::load(g, e) * v[j]);
    }
  }
}

// fp32 backward on the fp32 tile layout (see fp32 tiles above).
template <int BITS>
__device__ inline u32x4_t grad32_half(u32x4_t g, uint32_t f, const Values<BITS>& val) {
  constexpr uint32_t kMask = (1u << BITS) - 1u;
  u32x4_t out;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    out[j] = __float_as_uint(__uint_as_float(g[j]) * val((f >> (BITS * j)) & kMask));
  return out;
}

template <int BITS>
__global__ __launch_bounds__(FEWBIT_BWD32_THREADS) void bwd32_kernel(
    const float* g, const uint32_t* __restrict__ codes, float* gin, int64_t n, int64_t nwords,
    TableArgs tab) {
  constexpr int U = FEWBIT_BWD32_UNROLL;
  constexpr int kWords = Codes32<BITS>::kWords;
  constexpr uint32_t kMask = (1u << BITS) - 1u;
  const WaveIndex wi = wave_index<FEWBIT_BWD32_THREADS>();
  const Values<BITS> val(tab);
  const int64_t full = n / kTile;
  const int64_t groups = full / U;
  const int64_t lane_off = static_cast<int64_t>(wi.lane) * 4;
  const uint32_t lane_b = static_cast<uint32_t>(wi.lane) * kLaneBytes;

  for (int64_t gi = wi.wave; gi < groups; gi += wi.nwaves) {
    const int64_t t0 = gi * U;
    u32x4_t in[U][2];
    uint32_t f[U][2];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        in[u][h] = Span(g + (t0 + u) * kTile + h * 256, kSpanBytes).ld16(lane_b);
        f[u][h] = load_field32<BITS, true>(Span(codes + (t0 + u) * kWords, kWords * 4), h, wi.lane, kWords);
      }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        Span(gin + (t0 + u) * kTile + h * 256, kSpanBytes).st16(lane_b, grad32_half<BITS>(in[u][h], f[u][h], val));
  }
  for (int64_t t = groups * U + wi.wave; t < full; t += wi.nwaves) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const u32x4_t in = Span(g + t * kTile + h * 256, kSpanBytes).ld16(lane_b);
      const uint32_t f = load_field32<BITS, true>(Span(codes + t * kWords, kWords * 4), h, wi.lane, kWords);
      Span(gin + t * kTile + h * 256, kSpanBytes).st16(lane_b, grad32_half<BITS>(in, f, val));
    }
  }
  if (n % kTile != 0 && wi.wave == full % wi.nwaves) {
    const int64_t t = full;
    const int64_t wbase = t * kWords;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t f = load_field32<BITS, false>(Span(codes + wbase, kWords * 4), h, wi.lane, nwords - wbase);
      float v[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) v[j] = val((f >> (BITS * j)) & kMask);   // all lanes
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t e = t * kTile + h * 256 + lane_off + j;
        if (e < n) gin[e] = g[e] * v[j];
      }
    }
  }
}

// ---------------------------------------------------------------- host side
int check_table(const fewbit_table* t) {
  if (!t) return FEWBIT_E_NULL;
  if (t->bits < 1 || t->bits > 4) return FEWBIT_E_BITS;
  if (t->act < FEWBIT_GELU || t->act > FEWBIT_SOFTPLUS) return FEWBIT_E_INVALID;
  constexpr int32_t kFlags = FEWBIT_FLAG_SYMMETRIC | FEWBIT_FLAG_TABLE_FWD | FEWBIT_FLAG_ELEMENT_FWD;
  if ((t->flags & ~kFlags) != 0 || t->reserved != 0) return FEWBIT_E_INVALID;
  if ((t->flags & FEWBIT_FLAG_TABLE_FWD) && (t->flags & FEWBIT_FLAG_ELEMENT_FWD)) return FEWBIT_E_INVALID;
  const int K = 1 << t->bits;
  for (int m = 0; m < K - 1; ++m) {
    if (!std::isfinite(t->s[m])) return FEWBIT_E_NUMERIC;
    if (m > 0 && !(t->s[m - 1] < t->s[m])) return FEWBIT_E_NUMERIC;
  }
  for (int m = 0; m < K; ++m)
    if (!std::isfinite(t->v[m])) return FEWBIT_E_NUMERIC;
  return FEWBIT_OK;
}

bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

TableArgs table_args(const fewbit_table* t) {
  TableArgs a;
  const int K = 1 << t->bits;
  for (int m = 0; m < 15; ++m) a.s[m] = (m < K - 1) ? t->s[m] : INFINITY;
  for (int m = 0; m < 16; ++m) a.v[m] = (m < K) ? t->v[m] : 0.0f;
  return a;
}

// Compute units of the current device, read once per device.
int device_cus() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = -1;
  if (dev >= 0 && dev < 64) {
    const int c = cache[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int c = 0;
  if (dev < 0 ||
      hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      c <= 0)
    c = 256;
  if (dev >= 0 && dev < 64) cache[dev].store(c, std::memory_order_relaxed);
  return c;
}

// Workgroups for n elements when each has `waves_per_block` streaming waves
// that take `unroll` tiles per loop trip: one tile group per wave at most,
// capped at wg_per_cu per compute unit when wg_per_cu > 0, and at 2^30
// workgroups in any case (beyond 2^42 or so elements, far more than device
// memory holds); every kernel's waves walk the tile groups, so a capped grid
// still covers all of them.
dim3 grid_for(int64_t n, int waves_per_block, int wg_per_cu, int unroll) {
  constexpr int64_t kMaxBlocks = int64_t{1} << 30;
  const int64_t tiles = n / kTile + (n % kTile != 0);
  const int64_t groups = (tiles + unroll - 1) / unroll;
  int64_t blocks = (groups + waves_per_block - 1) / waves_per_block;
  if (wg_per_cu > 0) {
    const int64_t cap = static_cast<int64_t>(device_cus()) * wg_per_cu;
    if (blocks > cap) blocks = cap;
  }
  if (blocks > kMaxBlocks) blocks = kMaxBlocks;
  if (blocks < 1) blocks = 1;
  return dim3(static_cast<unsigned>(blocks));
}

// The stream must belong to the current device: the grid size, the output
// tables and the launch all refer to the current device.
int check_stream_device(hipStream_t stream) {
  int current = 0;
  hipDevice_t owner = 0;
  if (hipGetDevice(&current) != hipSuccess || hipStreamGetDevice(stream, &owner) != hipSuccess)
    return FEWBIT_E_HIP;
  return owner == current ? FEWBIT_OK : FEWBIT_E_INVALID;
}

struct Launch {
  const fewbit_table* t;
  const void* in;
  void* out;
  uint32_t* codes;
  int64_t n;
  hipStream_t s;
};

// The output-table runs of (ACT, DT) as a kernel argument; unused entries
// start past the last block.
template <int DT, int ACT>
OutRuns out_runs() {
  const fwd16_rules::Runs& src = fwd16_rules::kRuns[ACT][DT == FEWBIT_BF16 ? 1 : 0];
  OutRuns r;
  for (int j = 0; j < fwd16_rules::kMaxRuns; ++j) r.r[j] = j < src.count ? src.r[j] : fwd16_rules::kUnused;
  return r;
}

// log2 of the element count from which an fp16 / bf16 forward runs the table
// kernel, by [type: fp16, bf16][activation][bits - 1]; 63: never.  The table
// kernel builds its tables in every workgroup (7-10 us of fixed cost for
// bf16, 12-15 us for fp16, whose tables need f in far more blocks) and runs
// as a persistent grid, which streams at about 72% of the HBM peak; the
// per-element kernel has no setup and a grid of two-tile waves that streams
// at up to 79%, but evaluates f and the compares per element.  Measured on
// MI355X (x ~ N(0, 1), 2^23 .. 2^28 elements, back-to-back launches, the
// mean after the first quarter): the table kernel from the size where it is
// ahead at every larger size measured (within 2%).  At 2^28 elements the
// per-element kernel of 1- and 2-bit codes is 4-8% ahead in such runs, but
// its rate under sustained load swings by about 15% (it draws more power),
// while the table kernel's holds: there the table kernel is used (28).
// Softplus, whose per-element f is the most expensive, switches first.
constexpr uint8_t kTableMinLog2[2][FEWBIT_SOFTPLUS + 1][4] = {
    {   // fp16
        {28, 28, 26, 27},   // gelu
        {28, 28, 27, 27},   // silu
        {28, 63, 26, 27},   // sigmoid
        {28, 27, 25, 25},   // tanh
        {28, 28, 28, 63},   // relu
        {28, 26, 25, 26},   // selu
        {28, 28, 25, 26},   // softplus
    },
    {   // bf16
        {28, 28, 24, 24},   // gelu
        {28, 28, 25, 26},   // silu
        {28, 28, 28, 27},   // sigmoid
        {28, 28, 24, 25},   // tanh
        {28, 28, 28, 28},   // relu
        {28, 28, 25, 27},   // selu
        {28, 28, 24, 24},   // softplus
    },
};

int64_t table_min_of(int dt, int act, int bits) {
  const int lg = kTableMinLog2[dt == FEWBIT_BF16 ? 1 : 0][act][bits - 1];
  return lg >= 63 ? INT64_MAX : int64_t{1} << lg;
}

template <int DT, int BITS, int ACT>
void launch_fwd(const Launch& L) {
  const int64_t nw = fewbit_packed_words(L.n, BITS);
  const int sym = (L.t->flags & FEWBIT_FLAG_SYMMETRIC) ? 1 : 0;
  if constexpr (DT == FEWBIT_F32) {
    const dim3 grid = grid_for(L.n, FEWBIT_FWD32_THREADS / kWave, FEWBIT_FWD32_WG_PER_CU, FEWBIT_FWD32_UNROLL);
    (void)hipGetLastError();
    hipLaunchKernelGGL((fwd32_kernel<BITS, ACT>), grid, dim3(FEWBIT_FWD32_THREADS), 0, L.s,
                       static_cast<const float*>(L.in), static_cast<float*>(L.out), L.codes, L.n,
                       nw, table_args(L.t), sym);
  } else {
    const bool table = (L.t->flags & FEWBIT_FLAG_TABLE_FWD) ||
                       (!(L.t->flags & FEWBIT_FLAG_ELEMENT_FWD) && L.n >= table_min_of(DT, ACT, BITS));
    if (!table) {
      const dim3 grid = grid_for(L.n, FEWBIT_FWD16V_THREADS / kWave, 0, FEWBIT_FWD16V_UNROLL);
      (void)hipGetLastError();
      hipLaunchKernelGGL((fwd16v_kernel<DT, BITS, ACT>), grid, dim3(FEWBIT_FWD16V_THREADS), 0, L.s,
                         static_cast<const uint16_t*>(L.in), static_cast<uint16_t*>(L.out), L.codes,
                         L.n, nw, table_args(L.t), sym);
    } else {
      const dim3 grid = grid_for(L.n, FEWBIT_FWD16_THREADS / kWave, FEWBIT_FWD16_WG_PER_CU, FEWBIT_FWD16_UNROLL);
      (void)hipGetLastError();
      hipLaunchKernelGGL((fwd16_kernel<DT, BITS, ACT>), grid, dim3(FEWBIT_FWD16_THREADS), 0, L.s,
                         static_cast<const uint16_t*>(L.in), static_cast<uint16_t*>(L.out), L.codes,
                         L.n, nw, table_args(L.t), sym, out_runs<DT, ACT>());
    }
  }
}

template <int DT, int BITS>
void launch_fwd_act(const Launch& L) {
  switch (L.t->act) {
    case FEWBIT_GELU: launch_fwd<DT, BITS, FEWBIT_GELU>(L); break;
    case FEWBIT_SILU: launch_fwd<DT, BITS, FEWBIT_SILU>(L); break;
    case FEWBIT_SIGMOID: launch_fwd<DT, BITS, FEWBIT_SIGMOID>(L); break;
    case FEWBIT_TANH: launch_fwd<DT, BITS, FEWBIT_TANH>(L); break;
    case FEWBIT_RELU: launch_fwd<DT, BITS, FEWBIT_RELU>(L); break;
    case FEWBIT_SELU: launch_fwd<DT, BITS, FEWBIT_SELU>(L); break;
    default: launch_fwd<DT, BITS, FEWBIT_SOFTPLUS>(L); break;
  }
}

template <int DT>
void launch_fwd_bits(const Launch& L) {
  switch (L.t->bits) {
    case 1: launch_fwd_act<DT, 1>(L); break;
    case 2: launch_fwd_act<DT, 2>(L); break;
    case 3: launch_fwd_act<DT, 3>(L); break;
    default: launch_fwd_act<DT, 4>(L); break;
  }
}

template <int DT, int BITS>
void launch_bwd(const Launch& L) {
  const int64_t nw = fewbit_packed_words(L.n, BITS);
  (void)hipGetLastError();
  if constexpr (DT == FEWBIT_F32) {
    const dim3 grid = grid_for(L.n, FEWBIT_BWD32_THREADS / kWave, 0, FEWBIT_BWD32_UNROLL);
    hipLaunchKernelGGL((bwd32_kernel<BITS>), grid, dim3(FEWBIT_BWD32_THREADS), 0, L.s,
                       static_cast<const float*>(L.in), L.codes, static_cast<float*>(L.out), L.n,
                       nw, table_args(L.t));
  } else {
    // one-wave workgroups: a whole number of runs of the tile order over the
    // full tiles, and one more workgroup when the partial tile's unit lies past them
    const int64_t full = L.n / kTile, run = BwdOrder<BITS>::kRun;
    int64_t units = (full + run - 1) / run * run;
    if (L.n % kTile != 0 && units <= BwdOrder<BITS>::unit_of_tile(full)) units = BwdOrder<BITS>::unit_of_tile(full) + 1;
    const dim3 grid = grid_for(units * kTile, 1, 0, 1);
    hipLaunchKernelGGL((bwd_kernel<DT, BITS>), grid, dim3(kWave), 0, L.s,
                       static_cast<const uint16_t*>(L.in), L.codes, static_cast<uint16_t*>(L.out),
                       L.n, nw, table_args(L.t));
  }
}

template <int DT>
void launch_bwd_bits(const Launch& L) {
  switch (L.t->bits) {
    case 1: launch_bwd<DT, 1>(L); break;
    case 2: launch_bwd<DT, 2>(L); break;
    case 3: launch_bwd<DT, 3>(L); break;
    default: launch_bwd<DT, 4>(L); break;
  }
}

// Status of the launch just made (the runtime's last-error slot was cleared
// right before it); with FEWBIT_DEBUG set in the environment the HIP error
// behind FEWBIT_E_HIP is printed to stderr.
int launch_status(const char* where) {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return FEWBIT_OK;
  if (std::getenv("FEWBIT_DEBUG"))
    std::fprintf(stderr, "fewbit: %s launch failed: %s (%s)\n", where, hipGetErrorName(e),
                 hipGetErrorString(e));
  return FEWBIT_E_HIP;
}

}  // namespace

extern "C" int fewbit_fwd(const fewbit_table* t, int32_t dtype, const void* x, void* y,
                          uint32_t* codes, int64_t n, void* stream) {
  int rc = check_table(t);
  if (rc != FEWBIT_OK) return rc;
  if (dtype < FEWBIT_F32 || dtype > FEWBIT_BF16) return FEWBIT_E_DTYPE;
  if (n < 0) return FEWBIT_E_INVALID;
  if (n == 0) return FEWBIT_OK;
  if (!x || !y || !codes) return FEWBIT_E_NULL;
  if (misaligned(x) || misaligned(y) || misaligned(codes)) return FEWBIT_E_ALIGN;
  rc = check_stream_device(static_cast<hipStream_t>(stream));
  if (rc != FEWBIT_OK) return rc;
  const Launch L{t, x, y, codes, n, static_cast<hipStream_t>(stream)};
  switch (dtype) {
    case FEWBIT_F32: launch_fwd_bits<FEWBIT_F32>(L); break;
    case FEWBIT_F16: launch_fwd_bits<FEWBIT_F16>(L); break;
    default: launch_fwd_bits<FEWBIT_BF16>(L); break;
  }
  return launch_status("fewbit_fwd");
}

extern "C" int64_t fewbit_fwd16_table_min(int32_t act, int32_t bits, int32_t dtype) {
  if (act < FEWBIT_GELU || act > FEWBIT_SOFTPLUS || bits < 1 || bits > 4 ||
      (dtype != FEWBIT_F16 && dtype != FEWBIT_BF16))
    return -1;
  return table_min_of(dtype, act, bits);
}

extern "C" int fewbit_bwd(const fewbit_table* t, int32_t dtype, const void* grad_out,
                          const uint32_t* codes, void* grad_in, int64_t n, void* stream) {
  int rc = check_table(t);
  if (rc != FEWBIT_OK) return rc;
  if (dtype < FEWBIT_F32 || dtype > FEWBIT_BF16) return FEWBIT_E_DTYPE;
  if (n < 0) return FEWBIT_E_INVALID;
  if (n == 0) return FEWBIT_OK;
  if (!grad_out || !codes || !grad_in) return FEWBIT_E_NULL;
  if (misaligned(grad_out) || misaligned(codes) || misaligned(grad_in)) return FEWBIT_E_ALIGN;
  rc = check_stream_device(static_cast<hipStream_t>(stream));
  if (rc != FEWBIT_OK) return rc;
  const Launch L{t, grad_out, grad_in, const_cast<uint32_t*>(codes), n,
                 static_cast<hipStream_t>(stream)};
  switch (dtype) {
    case FEWBIT_F32: launch_bwd_bits<FEWBIT_F32>(L); break;
    case FEWBIT_F16: launch_bwd_bits<FEWBIT_F16>(L); break;
    default: launch_bwd_bits<FEWBIT_BF16>(L); break;
  }
  return launch_status("fewbit_bwd");
}

extern "C" const char* fewbit_strerror(int32_t status) {
  switch (status) {
    case FEWBIT_OK: return "success";
    case FEWBIT_E_INVALID: return "invalid argument";
    case FEWBIT_E_NULL: return "null pointer";
    case FEWBIT_E_ALIGN: return "pointer not 16-byte aligned";
    case FEWBIT_E_DTYPE: return "unknown storage type";
    case FEWBIT_E_BITS: return "bits must be 1..4";
    case FEWBIT_E_NOMEM: return "host allocation failed";
    case FEWBIT_E_NUMERIC: return "table boundaries not strictly increasing or not finite";
    case FEWBIT_E_HIP: return "HIP launch failed";
  }
  return "unknown status";
}
