// fewbit.hip -- gfx950 kernels and C ABI of the few-bit activation path.
//
// Forward (Listing 1, forward; Eq. (2)): y = f(x) plus, for every element,
// the index of the interval of the piecewise-constant approximation of f'
// it falls in, packed densely at `bits` bits per element.
// Backward (Eq. (1) with f' replaced by the approximation; Listing 1,
// backward): grad_in = grad_out * v[idx].
//
// Both passes are pointwise and bound by HBM bandwidth.  Work is cut into
// wave tiles of 512 consecutive elements: each of the 64 lanes of a wave
// owns 8 consecutive elements (one 16-byte access for fp16/bf16, two for
// fp32).  Eight codes of b bits make a b-byte field per lane, so the codes
// of a tile are exactly 16*b whole words and the fields of 4 neighbouring
// lanes (one DPP quad) always cover whole words: lanes combine their fields
// with quad permutes instead of atomics or shared memory, and every packed
// word has exactly one writer.
//
// The table (boundaries s, values v) travels as kernel arguments, i.e. in
// scalar registers; the backward mirrors v into LDS for per-lane lookup.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>

#include "../../include/fewbit.h"

namespace {

constexpr int kWave = 64;
constexpr int kPerLane = 8;                 // elements per lane per tile
constexpr int kTile = kWave * kPerLane;     // 512 elements per wave tile
constexpr int kBlock = 256;                 // 4 waves per workgroup
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int64_t kMaxBlocks = 256 * 8;     // 8 resident workgroups per CU

struct TableArgs {
  float s[15];
  float v[16];
};

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------- storage
template <int DT>
struct Storage;

template <>
struct Storage<FEWBIT_F32> {
  __device__ static void load8(const void* p, int64_t e, float (&f)[8]) {
    const float4* q = reinterpret_cast<const float4*>(static_cast<const float*>(p) + e);
    const float4 a = q[0], b = q[1];
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
    f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
  __device__ static void store8(void* p, int64_t e, const float (&f)[8]) {
    float4* q = reinterpret_cast<float4*>(static_cast<float*>(p) + e);
    q[0] = make_float4(f[0], f[1], f[2], f[3]);
    q[1] = make_float4(f[4], f[5], f[6], f[7]);
  }
  __device__ static float load1(const void* p, int64_t e) {
    return static_cast<const float*>(p)[e];
  }
  __device__ static void store1(void* p, int64_t e, float v) {
    static_cast<float*>(p)[e] = v;
  }
};

// bfloat16 is the upper half of a binary32: widening is a shift; narrowing
// rounds to nearest even (v_cvt_pk_bf16_f32 on gfx950).
template <>
struct Storage<FEWBIT_BF16> {
  __device__ static float lo(uint32_t u) { return __uint_as_float(u << 16); }
  __device__ static float hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }
  __device__ static uint32_t pack(float a, float b) {
    const bf16x2_t h = __builtin_convertvector((f32x2_t){a, b}, bf16x2_t);
    return __builtin_bit_cast(uint32_t, h);
  }
  __device__ static void load8(const void* p, int64_t e, float (&f)[8]) {
    const uint4 u = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p) + e);
    f[0] = lo(u.x); f[1] = hi(u.x); f[2] = lo(u.y); f[3] = hi(u.y);
    f[4] = lo(u.z); f[5] = hi(u.z); f[6] = lo(u.w); f[7] = hi(u.w);
  }
  __device__ static void store8(void* p, int64_t e, const float (&f)[8]) {
    uint4 u;
    u.x = pack(f[0], f[1]); u.y = pack(f[2], f[3]);
    u.z = pack(f[4], f[5]); u.w = pack(f[6], f[7]);
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(p) + e) = u;
  }
  __device__ static float load1(const void* p, int64_t e) {
    return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(p)[e]) << 16);
  }
  __device__ static void store1(void* p, int64_t e, float v) {
    static_cast<uint16_t*>(p)[e] = static_cast<uint16_t>(pack(v, 0.0f) & 0xFFFFu);
  }
};

template <>
struct Storage<FEWBIT_F16> {
  __device__ static uint32_t pack(float a, float b) {
    const f16x2_t h = __builtin_convertvector((f32x2_t){a, b}, f16x2_t);
    return __builtin_bit_cast(uint32_t, h);
  }
  __device__ static void unpack(uint32_t u, float& a, float& b) {
    const f16x2_t h = __builtin_bit_cast(f16x2_t, u);
    a = static_cast<float>(h.x);
    b = static_cast<float>(h.y);
  }
  __device__ static void load8(const void* p, int64_t e, float (&f)[8]) {
    const uint4 u = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p) + e);
    unpack(u.x, f[0], f[1]); unpack(u.y, f[2], f[3]);
    unpack(u.z, f[4], f[5]); unpack(u.w, f[6], f[7]);
  }
  __device__ static void store8(void* p, int64_t e, const float (&f)[8]) {
    uint4 u;
    u.x = pack(f[0], f[1]); u.y = pack(f[2], f[3]);
    u.z = pack(f[4], f[5]); u.w = pack(f[6], f[7]);
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(p) + e) = u;
  }
  __device__ static float load1(const void* p, int64_t e) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<const uint16_t*>(p)[e]));
  }
  __device__ static void store1(void* p, int64_t e, float v) {
    static_cast<uint16_t*>(p)[e] = static_cast<uint16_t>(pack(v, 0.0f) & 0xFFFFu);
  }
};

// ---------------------------------------------------------------- activations
// Each f is evaluated in fp32.  The products x*Phi(x) and x*sigmoid(x) are
// formed as relu(x) - |x| * tail(|x|), with tail the upper tail probability
// (Q for the normal, sigmoid(-|x|) for the logistic), so the negative side
// keeps full relative accuracy down to the subnormal range.
template <int ACT>
struct Act;

template <>
struct Act<FEWBIT_GELU> {
  __device__ static float f(float x) {
    const float t = fabsf(x);
    const float q = 0.5f * erfcf(t * 0.70710678118654752f);   // P(Z > |x|)
    float y = (x >= 0.0f) ? fmaf(-x, q, x) : x * q;
    if (__builtin_isinf(x)) y = (x > 0.0f) ? x : -0.0f;
    return y;
  }
};

template <>
struct Act<FEWBIT_SILU> {
  __device__ static float f(float x) {
    const float t = fabsf(x);
    const float e = expf(-t);
    const float tail = e / (1.0f + e);                          // sigmoid(-|x|)
    float y = (x >= 0.0f) ? fmaf(-x, tail, x) : x * tail;
    if (__builtin_isinf(x)) y = (x > 0.0f) ? x : -0.0f;
    return y;
  }
};

template <>
struct Act<FEWBIT_SIGMOID> {
  __device__ static float f(float x) {
    const float e = expf(-fabsf(x));
    const float r = 1.0f / (1.0f + e);                          // sigmoid(|x|)
    return (x >= 0.0f) ? r : (x < 0.0f ? e * r : x);            // NaN -> NaN
  }
};

template <>
struct Act<FEWBIT_TANH> {
  __device__ static float f(float x) { return tanhf(x); }
};

// ---------------------------------------------------------------- classify
// idx = number of boundaries s[m] <= x: half-open intervals [s[m-1], s[m]).
// IEEE compares: NaN gives 0, -0 == +0, subnormals are not flushed.
template <int BITS>
__device__ inline uint32_t classify(float x, const TableArgs& tab) {
  uint32_t c = 0;
#pragma unroll
  for (int m = 0; m < (1 << BITS) - 1; ++m) c += (x >= tab.s[m]) ? 1u : 0u;
  return c;
}

// ---------------------------------------------------------------- packing
// quad_perm DPP control: lane k of each quad reads lane sel[k] of the quad.
constexpr int quad_perm(int a, int b, int c, int d) { return a | (b << 2) | (c << 4) | (d << 6); }

template <int CTRL>
__device__ inline uint32_t quad_read(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), CTRL, 0xF, 0xF, false));
}

// Lane field F holds the 8 codes of the lane (8*BITS bits, code j at bit
// BITS*j).  The tile's stream is the lane fields laid end to end, so lane l's
// field starts at stream bit 8*BITS*l.  Writes the words of the tile whose
// index is below `valid` (the rest belong past the end of the buffer).
// Must be called by all 64 lanes together.
template <int BITS>
__device__ inline void pack_store(uint32_t* out, uint32_t F, int lane, int64_t valid) {
  if constexpr (BITS == 4) {
    if (lane < valid) out[lane] = F;
  } else if constexpr (BITS == 2) {
    const uint32_t nb = quad_read<quad_perm(1, 1, 3, 3)>(F);
    const uint32_t w = F | (nb << 16);
    const int widx = lane >> 1;
    if (!(lane & 1) && widx < valid) out[widx] = w;
  } else if constexpr (BITS == 1) {
    const uint32_t n1 = quad_read<quad_perm(1, 1, 3, 3)>(F);
    const uint32_t a = F | (n1 << 8);
    const uint32_t n2 = quad_read<quad_perm(2, 2, 2, 2)>(a);
    const uint32_t w = a | (n2 << 16);
    const int widx = lane >> 2;
    if (!(lane & 3) && widx < valid) out[widx] = w;
  } else {  // BITS == 3: a quad's 4 x 24 bits are words 3q, 3q+1, 3q+2
    const uint32_t nx = quad_read<quad_perm(1, 2, 3, 3)>(F);
    const int k = lane & 3;
    const uint32_t w = (F >> (8 * k)) | (nx << (24 - 8 * k));
    const int widx = 3 * (lane >> 2) + k;
    if (k < 3 && widx < valid) out[widx] = w;
  }
}

// Inverse of the layout above: the lane's 8*BITS-bit field.
template <int BITS>
__device__ inline uint32_t load_field(const uint32_t* base, int lane, int64_t valid) {
  const int bit = 8 * BITS * lane;
  const int w = bit >> 5, sh = bit & 31;
  const uint32_t lo = (w < valid) ? base[w] : 0u;
  if (sh + 8 * BITS > 32) {
    const uint32_t hi = (w + 1 < valid) ? base[w + 1] : 0u;
    return __builtin_amdgcn_alignbit(hi, lo, sh);
  }
  return lo >> sh;
}

// ---------------------------------------------------------------- kernels
template <int DT, int BITS, int ACT>
__global__ __launch_bounds__(kBlock) void fwd_kernel(const void* x, void* y,
                                                     uint32_t* __restrict__ codes,
                                                     int64_t n, int64_t nwords,
                                                     TableArgs tab, int symmetric) {
  using S = Storage<DT>;
  constexpr int kWordsPerTile = 16 * BITS;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
  const int64_t nwaves = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
  const int64_t full = n / kTile;

  for (int64_t t = wave; t < full; t += nwaves) {
    const int64_t e = t * kTile + static_cast<int64_t>(lane) * kPerLane;
    float xf[8], yf[8];
    S::load8(x, e, xf);
    uint32_t F = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      yf[j] = Act<ACT>::f(xf[j]);
      const float xc = symmetric ? fabsf(xf[j]) : xf[j];
      F |= classify<BITS>(xc, tab) << (BITS * j);
    }
    S::store8(y, e, yf);
    pack_store<BITS>(codes + t * kWordsPerTile, F, lane, kWordsPerTile);
  }

  // the partial tile at the end, if any, goes to the wave that would own it
  if (n % kTile != 0 && wave == full % nwaves) {
    const int64_t t = full;
    uint32_t F = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t e = t * kTile + static_cast<int64_t>(lane) * kPerLane + j;
      if (e < n) {
        const float xv = S::load1(x, e);
        S::store1(y, e, Act<ACT>::f(xv));
        const float xc = symmetric ? fabsf(xv) : xv;
        F |= classify<BITS>(xc, tab) << (BITS * j);
      }
    }
    const int64_t wbase = t * kWordsPerTile;
    pack_store<BITS>(codes + wbase, F, lane, nwords - wbase);
  }
}

template <int DT, int BITS>
__global__ __launch_bounds__(kBlock) void bwd_kernel(const void* g,
                                                     const uint32_t* __restrict__ codes,
                                                     void* gin, int64_t n, int64_t nwords,
                                                     TableArgs tab) {
  using S = Storage<DT>;
  constexpr int kWordsPerTile = 16 * BITS;
  constexpr uint32_t kMask = (1u << BITS) - 1u;
  __shared__ float val[16];
  if (threadIdx.x < 16) val[threadIdx.x] = tab.v[threadIdx.x];
  __syncthreads();

  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
  const int64_t nwaves = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
  const int64_t full = n / kTile;

  for (int64_t t = wave; t < full; t += nwaves) {
    const int64_t e = t * kTile + static_cast<int64_t>(lane) * kPerLane;
    float gf[8];
    S::load8(g, e, gf);
    const uint32_t F = load_field<BITS>(codes + t * kWordsPerTile, lane, kWordsPerTile);
#pragma unroll
    for (int j = 0; j < 8; ++j) gf[j] = gf[j] * val[(F >> (BITS * j)) & kMask];
    S::store8(gin, e, gf);
  }

  if (n % kTile != 0 && wave == full % nwaves) {
    const int64_t t = full;
    const int64_t wbase = t * kWordsPerTile;
    const uint32_t F = load_field<BITS>(codes + wbase, lane, nwords - wbase);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t e = t * kTile + static_cast<int64_t>(lane) * kPerLane + j;
      if (e < n) S::store1(gin, e, S::load1(g, e) * val[(F >> (BITS * j)) & kMask]);
    }
  }
}

// ---------------------------------------------------------------- host side
int check_table(const fewbit_table* t) {
  if (!t) return FEWBIT_E_NULL;
  if (t->bits < 1 || t->bits > 4) return FEWBIT_E_BITS;
  if (t->act < FEWBIT_GELU || t->act > FEWBIT_TANH) return FEWBIT_E_INVALID;
  if ((t->flags & ~FEWBIT_FLAG_SYMMETRIC) != 0 || t->reserved != 0) return FEWBIT_E_INVALID;
  const int K = 1 << t->bits;
  for (int m = 0; m < K - 1; ++m) {
    if (!std::isfinite(t->s[m])) return FEWBIT_E_NUMERIC;
    if (m > 0 && !(t->s[m - 1] < t->s[m])) return FEWBIT_E_NUMERIC;
  }
  for (int m = 0; m < K; ++m)
    if (!std::isfinite(t->v[m])) return FEWBIT_E_NUMERIC;
  return FEWBIT_OK;
}

// Status of the launch just made; with FEWBIT_DEBUG set in the environment
// the HIP error behind FEWBIT_E_HIP is printed to stderr.
int launch_status(const char* where) {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return FEWBIT_OK;
  if (std::getenv("FEWBIT_DEBUG"))
    std::fprintf(stderr, "fewbit: %s launch failed: %s (%s)\n", where, hipGetErrorName(e),
                 hipGetErrorString(e));
  return FEWBIT_E_HIP;
}

bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

TableArgs table_args(const fewbit_table* t) {
  TableArgs a;
  const int K = 1 << t->bits;
  for (int m = 0; m < 15; ++m) a.s[m] = (m < K - 1) ? t->s[m] : INFINITY;
  for (int m = 0; m < 16; ++m) a.v[m] = (m < K) ? t->v[m] : 0.0f;
  return a;
}

dim3 grid_for(int64_t n) {
  const int64_t tiles = (n + kTile - 1) / kTile;
  int64_t blocks = (tiles + kWavesPerBlock - 1) / kWavesPerBlock;
  if (blocks > kMaxBlocks) blocks = kMaxBlocks;
  if (blocks < 1) blocks = 1;
  return dim3(static_cast<unsigned>(blocks));
}

template <int DT, int BITS, int ACT>
void launch_fwd(const fewbit_table* t, const void* x, void* y, uint32_t* codes, int64_t n,
                hipStream_t s) {
  const int64_t nw = (n * BITS + 31) / 32;
  hipLaunchKernelGGL((fwd_kernel<DT, BITS, ACT>), grid_for(n), dim3(kBlock), 0, s, x, y, codes,
                     n, nw, table_args(t), (t->flags & FEWBIT_FLAG_SYMMETRIC) ? 1 : 0);
}

template <int DT, int BITS>
void launch_fwd_act(const fewbit_table* t, const void* x, void* y, uint32_t* codes, int64_t n,
                    hipStream_t s) {
  switch (t->act) {
    case FEWBIT_GELU: launch_fwd<DT, BITS, FEWBIT_GELU>(t, x, y, codes, n, s); break;
    case FEWBIT_SILU: launch_fwd<DT, BITS, FEWBIT_SILU>(t, x, y, codes, n, s); break;
    case FEWBIT_SIGMOID: launch_fwd<DT, BITS, FEWBIT_SIGMOID>(t, x, y, codes, n, s); break;
    default: launch_fwd<DT, BITS, FEWBIT_TANH>(t, x, y, codes, n, s); break;
  }
}

template <int DT>
void launch_fwd_bits(const fewbit_table* t, const void* x, void* y, uint32_t* codes, int64_t n,
                     hipStream_t s) {
  switch (t->bits) {
    case 1: launch_fwd_act<DT, 1>(t, x, y, codes, n, s); break;
    case 2: launch_fwd_act<DT, 2>(t, x, y, codes, n, s); break;
    case 3: launch_fwd_act<DT, 3>(t, x, y, codes, n, s); break;
    default: launch_fwd_act<DT, 4>(t, x, y, codes, n, s); break;
  }
}

template <int DT, int BITS>
void launch_bwd(const fewbit_table* t, const void* g, const uint32_t* codes, void* gin, int64_t n,
                hipStream_t s) {
  const int64_t nw = (n * BITS + 31) / 32;
  hipLaunchKernelGGL((bwd_kernel<DT, BITS>), grid_for(n), dim3(kBlock), 0, s, g, codes, gin, n,
                     nw, table_args(t));
}

template <int DT>
void launch_bwd_bits(const fewbit_table* t, const void* g, const uint32_t* codes, void* gin,
                     int64_t n, hipStream_t s) {
  switch (t->bits) {
    case 1: launch_bwd<DT, 1>(t, g, codes, gin, n, s); break;
    case 2: launch_bwd<DT, 2>(t, g, codes, gin, n, s); break;
    case 3: launch_bwd<DT, 3>(t, g, codes, gin, n, s); break;
    default: launch_bwd<DT, 4>(t, g, codes, gin, n, s); break;
  }
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
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the runtime's last-error slot may hold an error left by an earlier,
  // unrelated call on this thread; clear it so the check below sees only
  // this launch
  (void)hipGetLastError();
  switch (dtype) {
    case FEWBIT_F32: launch_fwd_bits<FEWBIT_F32>(t, x, y, codes, n, s); break;
    case FEWBIT_F16: launch_fwd_bits<FEWBIT_F16>(t, x, y, codes, n, s); break;
    default: launch_fwd_bits<FEWBIT_BF16>(t, x, y, codes, n, s); break;
  }
  return launch_status("fewbit_fwd");
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
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();  // see fewbit_fwd
  switch (dtype) {
    case FEWBIT_F32: launch_bwd_bits<FEWBIT_F32>(t, grad_out, codes, grad_in, n, s); break;
    case FEWBIT_F16: launch_bwd_bits<FEWBIT_F16>(t, grad_out, codes, grad_in, n, s); break;
    default: launch_bwd_bits<FEWBIT_BF16>(t, grad_out, codes, grad_in, n, s); break;
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
