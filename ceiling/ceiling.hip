// ceiling.hip -- streaming reference kernels for the benchmark (not part of
// the few-bit library, never linked into it).
//
// They move exactly the bytes of the few-bit passes with nothing else to do,
// so their rate is what this device can stream for each byte mix: the
// practical ceiling the library kernels are compared against in the same run.
//
//   copy      read s*512 B, write s*512 B per 512-element tile
//   fwd mix   read s*512 B, write s*512 B + 16*b code words (the forward's
//             bytes: x in, y and the packed codes out)
//   bwd mix   read s*512 B + 16*b code words, write s*512 B (the backward's
//             bytes: grad_out and the codes in, grad_in out)
//
// s is the element size (2 or 4 bytes) and b the bits per code.  Every access
// is a 16-byte non-temporal buffer access whose wave instruction covers 1 KiB
// of contiguous memory, in the launch shapes that stream best on this device:
// one wave per tile, the hardware dispatcher handing out workgroups as earlier
// ones retire.  Only whole tiles are moved.
//
// At 1 and 3 bits a tile's code span is not a whole number of 128-byte
// lines, so tiles 2p and 2p+1 share a line.  Read by waves on two XCDs (whose
// L2 caches are separate) it is fetched twice; the paired launch shape gives
// the two tiles to one-wave workgroups 8 apart in launch order, which the
// dispatcher places on the same XCD, so the line is fetched once.
//
// One more shape stands for the 16-bit table forward's own launch: one
// persistent 512-thread workgroup per compute unit (LDS-bound, as the
// forward's 160 KiB of tables make it), wave w of W taking tiles w, w + W,
// w + 2W, ... with the loads of its next four tiles in flight.  It is not a
// candidate for the ceiling; it shows what that launch shape can stream.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ inline __amdgpu_buffer_rsrc_t span(const void* p, uint32_t bytes) {
  // 0x00020000: raw 32-bit buffer accesses (gfx9 descriptor word 3)
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, static_cast<int>(bytes), 0x00020000);
}
__device__ inline u32x4_t ld16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2);      // nt
}
__device__ inline void st16(__amdgpu_buffer_rsrc_t r, uint32_t off, u32x4_t v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, 2);
}

// workgroup u of a run of 16 takes tile 2 (u mod 8) + (u mod 16) / 8 of the run
__device__ inline int64_t paired_tile(int64_t u) {
  const int64_t r = u & 15;
  return (u - r) + 2 * (r & 7) + (r >> 3);
}

// KIND 0 copy, 1 forward mix, 2 backward mix; S element bytes.  Lane l moves
// bytes 16 l .. 16 l + 15 of each 1 KiB chunk of the tile (S / 2 chunks).
// The code words of a tile (16 b of them) are read or written by lane
// l mod 16 b: lanes past the last word repeat a lower lane's access, so no
// lane is masked off.
template <int KIND, int S, int TPB, bool PAIRED>
__global__ __launch_bounds__(TPB) void stream_kernel(const uint8_t* src, uint8_t* dst, uint32_t* codes,
                                                     int64_t tiles, int words, uint32_t salt) {
  constexpr uint32_t kTileBytes = 512u * S;
  const int lane = threadIdx.x & 63;
  const int64_t u = static_cast<int64_t>(blockIdx.x) * (TPB / 64) +
                    __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x / 64));
  const int64_t t = PAIRED ? paired_tile(u) : u;
  if (t >= tiles) return;
  const auto rs = span(src + t * kTileBytes, kTileBytes);
  const auto rd = span(dst + t * kTileBytes, kTileBytes);
  const auto rc = span(codes + t * words, static_cast<uint32_t>(words) * 4u);
  const uint32_t wo = static_cast<uint32_t>(lane % words) * 4u;
  u32x4_t v[S / 2];
#pragma unroll
  for (int h = 0; h < S / 2; ++h) v[h] = ld16(rs, h * 1024u + lane * 16u);
  uint32_t c = salt;
  if constexpr (KIND == 2) c ^= __builtin_amdgcn_raw_buffer_load_b32(rc, wo, 0, 2);
#pragma unroll
  for (int h = 0; h < S / 2; ++h) st16(rd, h * 1024u + lane * 16u, v[h] ^ c);
  if constexpr (KIND == 1) __builtin_amdgcn_raw_buffer_store_b32(v[0].x ^ v[0].y ^ salt, rc, wo, 0, 2);
}

// The persistent shape: per tile, the loads (data and, for the backward mix,
// the code word) and then the stores, as in stream_kernel.
template <int KIND, int S>
struct Loaded {
  u32x4_t v[S / 2];
  uint32_t c;
};
template <int KIND, int S>
__device__ inline Loaded<KIND, S> load_tile(const uint8_t* src, const uint32_t* codes, int64_t t, int64_t tiles,
                                            int words, int lane) {
  constexpr uint32_t kTileBytes = 512u * S;
  const bool in = t < tiles;
  const auto rs = span(src + (in ? t : 0) * kTileBytes, in ? kTileBytes : 0u);
  Loaded<KIND, S> r;
#pragma unroll
  for (int h = 0; h < S / 2; ++h) r.v[h] = ld16(rs, h * 1024u + lane * 16u);
  r.c = 0;
  if constexpr (KIND == 2) {
    const auto rc = span(codes + (in ? t : 0) * words, in ? static_cast<uint32_t>(words) * 4u : 0u);
    r.c = __builtin_amdgcn_raw_buffer_load_b32(rc, static_cast<uint32_t>(lane % words) * 4u, 0, 2);
  }
  return r;
}
template <int KIND, int S>
__device__ inline void store_tile(uint8_t* dst, uint32_t* codes, int64_t t, int words, int lane,
                                  const Loaded<KIND, S>& r, uint32_t salt) {
  constexpr uint32_t kTileBytes = 512u * S;
  const auto rd = span(dst + t * kTileBytes, kTileBytes);
  const uint32_t c = salt ^ r.c;
#pragma unroll
  for (int h = 0; h < S / 2; ++h) st16(rd, h * 1024u + lane * 16u, r.v[h] ^ c);
  if constexpr (KIND == 1) {
    const auto rc = span(codes + t * words, static_cast<uint32_t>(words) * 4u);
    __builtin_amdgcn_raw_buffer_store_b32(r.v[0].x ^ r.v[0].y ^ salt, rc, static_cast<uint32_t>(lane % words) * 4u,
                                          0, 2);
  }
}

constexpr int kPersistThreads = 512;
constexpr int kPersistDepth = 4;

template <int KIND, int S>
__global__ __launch_bounds__(kPersistThreads) void persist_kernel(const uint8_t* src, uint8_t* dst, uint32_t* codes,
                                                                  int64_t tiles, int words, uint32_t salt) {
  // 156 KiB of LDS: one workgroup per compute unit
  __shared__ uint32_t hold[156 * 1024 / 4];
  const int lane = threadIdx.x & 63;
  const int64_t w = static_cast<int64_t>(blockIdx.x) * (kPersistThreads / 64) +
                    __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x / 64));
  const int64_t nw = static_cast<int64_t>(gridDim.x) * (kPersistThreads / 64);
  if (threadIdx.x == 0) hold[0] = salt;
  __syncthreads();
  const uint32_t s = hold[0];
  Loaded<KIND, S> q[kPersistDepth];
#pragma unroll
  for (int d = 0; d < kPersistDepth; ++d) q[d] = load_tile<KIND, S>(src, codes, w + d * nw, tiles, words, lane);
  for (int64_t t = w; t < tiles; t += kPersistDepth * nw) {
#pragma unroll
    for (int d = 0; d < kPersistDepth; ++d) {
      const int64_t tt = t + d * nw;
      const Loaded<KIND, S> cur = q[d];
      q[d] = load_tile<KIND, S>(src, codes, tt + kPersistDepth * nw, tiles, words, lane);
      if (tt < tiles) store_tile<KIND, S>(dst, codes, tt, words, lane, cur, s);
    }
  }
}

template <int KIND, int S>
hipError_t launch_s(int shape, const void* src, void* dst, uint32_t* codes, int64_t tiles, int words,
                    hipStream_t s) {
  const auto* in = static_cast<const uint8_t*>(src);
  auto* out = static_cast<uint8_t*>(dst);
  (void)hipGetLastError();
  switch (shape) {
    case 64:
      hipLaunchKernelGGL((stream_kernel<KIND, S, 64, false>), dim3(static_cast<unsigned>(tiles)), dim3(64), 0,
                         s, in, out, codes, tiles, words, 0u);
      break;
    case 256:
      hipLaunchKernelGGL((stream_kernel<KIND, S, 256, false>), dim3(static_cast<unsigned>((tiles + 3) / 4)),
                         dim3(256), 0, s, in, out, codes, tiles, words, 0u);
      break;
    case 65:   // 64 threads, paired tile order: a whole number of runs of 16
      hipLaunchKernelGGL((stream_kernel<KIND, S, 64, true>), dim3(static_cast<unsigned>((tiles + 15) / 16 * 16)),
                         dim3(64), 0, s, in, out, codes, tiles, words, 0u);
      break;
    case 512: {   // persistent: one workgroup per compute unit
      int dev = 0, cus = 0;
      if (hipGetDevice(&dev) != hipSuccess ||
          hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        return hipErrorInvalidValue;
      hipLaunchKernelGGL((persist_kernel<KIND, S>), dim3(static_cast<unsigned>(cus)), dim3(kPersistThreads), 0, s,
                         in, out, codes, tiles, words, 0u);
      break;
    }
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

// Streams `tiles` whole 512-element tiles of kind 0 (copy), 1 (forward byte
// mix) or 2 (backward byte mix) of elem_bytes-byte elements (2 or 4) with
// bits-bit codes (1..4) on `stream`, in launch shape `shape`: 64 or 256
// threads per workgroup in tile order, 65: 64 threads in the paired order,
// or 512: persistent 512-thread workgroups, one per compute unit of the
// current device.
// src and dst hold tiles * 512 * elem_bytes bytes, codes tiles * 16 * bits
// words (unused for the copy); all 16-byte aligned.  Returns 0, or -1 for an
// argument error, -2 for a launch error.
extern "C" int ceiling_stream(int kind, int shape, int elem_bytes, int bits, const void* src, void* dst,
                              uint32_t* codes, int64_t tiles, void* stream) {
  if (kind < 0 || kind > 2 || (elem_bytes != 2 && elem_bytes != 4) || bits < 1 || bits > 4 ||
      tiles < 0 || tiles > (int64_t{1} << 31) - 16 || (shape != 64 && shape != 256 && shape != 65 && shape != 512))
    return -1;
  if (tiles == 0) return 0;
  if (!src || !dst || (kind != 0 && !codes)) return -1;
  const int words = 16 * bits;
  auto s = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (elem_bytes == 2) {
    e = kind == 0   ? launch_s<0, 2>(shape, src, dst, codes, tiles, words, s)
        : kind == 1 ? launch_s<1, 2>(shape, src, dst, codes, tiles, words, s)
                    : launch_s<2, 2>(shape, src, dst, codes, tiles, words, s);
  } else {
    e = kind == 0   ? launch_s<0, 4>(shape, src, dst, codes, tiles, words, s)
        : kind == 1 ? launch_s<1, 4>(shape, src, dst, codes, tiles, words, s)
                    : launch_s<2, 4>(shape, src, dst, codes, tiles, words, s);
  }
  return e == hipSuccess ? 0 : -2;
}
