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
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

// Streams `tiles` whole 512-element tiles of kind 0 (copy), 1 (forward byte
// mix) or 2 (backward byte mix) of elem_bytes-byte elements (2 or 4) with
// bits-bit codes (1..4) on `stream`, in launch shape `shape`: 64 or 256
// threads per workgroup in tile order, or 65: 64 threads in the paired order.
// src and dst hold tiles * 512 * elem_bytes bytes, codes tiles * 16 * bits
// words (unused for the copy); all 16-byte aligned.  Returns 0, or -1 for an
// argument error, -2 for a launch error.
extern "C" int ceiling_stream(int kind, int shape, int elem_bytes, int bits, const void* src, void* dst,
                              uint32_t* codes, int64_t tiles, void* stream) {
  if (kind < 0 || kind > 2 || (elem_bytes != 2 && elem_bytes != 4) || bits < 1 || bits > 4 ||
      tiles < 0 || tiles > (int64_t{1} << 31) - 16 || (shape != 64 && shape != 256 && shape != 65))
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
