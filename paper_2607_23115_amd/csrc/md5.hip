// gleam_md5_prefix: the paper's own chunk identifier (Appendix, discussion of hash
// cost and collisions): an MD5 string of the first 1024 bits (128 bytes) of each
// host-to-device chunk; chunks of at most 1024 bytes get no cache entry. Kept as an
// ablation of the full-content block digests: it reads 128 bytes per payload, but it
// cannot see a change past the prefix nor a repeat smaller than a payload.
//
// MD5 as specified in RFC 1321: pad with a 1 bit, zeros to 56 mod 64 bytes and the
// 64-bit little-endian bit length; per 64-byte block, four rounds of sixteen steps
// over the state (A, B, C, D). One lane per payload.

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

constexpr int kThreads = 256;
constexpr uint32_t kMaxPrefix = 1u << 20;

// RFC 1321, section 3.4: T[i] = floor(2^32 * |sin(i)|), i = 1..64.
__constant__ uint32_t kT[64] = {
    0xd76aa478, 0xe8c7b756, 0x242070db, 0xc1bdceee, 0xf57c0faf, 0x4787c62a, 0xa8304613, 0xfd469501,
    0x698098d8, 0x8b44f7af, 0xffff5bb1, 0x895cd7be, 0x6b901122, 0xfd987193, 0xa679438e, 0x49b40821,
    0xf61e2562, 0xc040b340, 0x265e5a51, 0xe9b6c7aa, 0xd62f105d, 0x02441453, 0xd8a1e681, 0xe7d3fbc8,
    0x21e1cde6, 0xc33707d6, 0xf4d50d87, 0x455a14ed, 0xa9e3e905, 0xfcefa3f8, 0x676f02d9, 0x8d2a4c8a,
    0xfffa3942, 0x8771f681, 0x6d9d6122, 0xfde5380c, 0xa4beea44, 0x4bdecfa9, 0xf6bb4b60, 0xbebfbc70,
    0x289b7ec6, 0xeaa127fa, 0xd4ef3085, 0x04881d05, 0xd9d4d039, 0xe6db99e5, 0x1fa27cf8, 0xc4ac5665,
    0xf4292244, 0x432aff97, 0xab9423a7, 0xfc93a039, 0x655b59c3, 0x8f0ccc92, 0xffeff47d, 0x85845dd1,
    0x6fa87e4f, 0xfe2ce6e0, 0xa3014314, 0x4e0811a1, 0xf7537e82, 0xbd3af235, 0x2ad7d2bb, 0xeb86d391};

__device__ __forceinline__ uint32_t rotl32(uint32_t x, int s) { return (x << s) | (x >> (32 - s)); }

__device__ __forceinline__ void md5_compress(uint32_t st[4], const uint32_t X[16]) {
  constexpr int kS[4][4] = {{7, 12, 17, 22}, {5, 9, 14, 20}, {4, 11, 16, 23}, {6, 10, 15, 21}};
  uint32_t a = st[0], b = st[1], c = st[2], d = st[3];
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    uint32_t f;
    int k;
    if (i < 16) {
      f = (b & c) | (~b & d);
      k = i;
    } else if (i < 32) {
      f = (b & d) | (c & ~d);
      k = (5 * i + 1) & 15;
    } else if (i < 48) {
      f = b ^ c ^ d;
      k = (3 * i + 5) & 15;
    } else {
      f = c ^ (b | ~d);
      k = (7 * i) & 15;
    }
    const uint32_t t = a + f + X[k] + kT[i];
    a = d;
    d = c;
    c = b;
    b = b + rotl32(t, kS[i >> 4][i & 3]);
  }
  st[0] += a;
  st[1] += b;
  st[2] += c;
  st[3] += d;
}

__global__ void md5_prefix_kernel(const uint64_t* seg_addr, const uint64_t* seg_len, uint64_t n_seg,
                                  uint32_t prefix, uint64_t min_len, uint64_t* digest, uint64_t* key,
                                  uint8_t* eligible) {
  const uint64_t s = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= n_seg) return;
  const uint64_t len = seg_len[s];
  const uint32_t L = len < prefix ? (uint32_t)len : prefix;
  const uint8_t* p = reinterpret_cast<const uint8_t*>(seg_addr[s]);
  const uint32_t blocks = (L + 8) / 64 + 1;
  const uint64_t bits = (uint64_t)L * 8;
  uint32_t st[4] = {0x67452301u, 0xefcdab89u, 0x98badcfeu, 0x10325476u};
  for (uint32_t blk = 0; blk < blocks; ++blk) {
    const uint32_t base = blk * 64;
    uint32_t X[16];
    if (base + 64 <= L) {
      // whole 64-byte block: 4-byte loads at any alignment (gfx950 under HSA runs with
      // unaligned access enabled), each inside the prefix
      typedef uint32_t u32_any __attribute__((aligned(1)));
#pragma unroll
      for (int w = 0; w < 16; ++w) X[w] = reinterpret_cast<const u32_any*>(p + base)[w];
    } else {
#pragma unroll
      for (int w = 0; w < 16; ++w) {
        uint32_t v = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t q = base + 4 * w + i;
          const uint32_t byte = q < L ? p[q] : (q == L ? 0x80u : 0u);
          v |= byte << (8 * i);
        }
        X[w] = v;
      }
      if (blk == blocks - 1) {
        X[14] = (uint32_t)bits;
        X[15] = (uint32_t)(bits >> 32);
      }
    }
    md5_compress(st, X);
  }
  const uint64_t lo = ((uint64_t)st[1] << 32) | st[0];
  const uint64_t hi = ((uint64_t)st[3] << 32) | st[2];
  digest[2 * s] = lo;
  digest[2 * s + 1] = hi;
  if (key) key[s] = lo;
  if (eligible) eligible[s] = len > min_len ? 1 : 0;
}

}  // namespace
// Loads this file's GPU code object on the current device (gleam_preload).
hipError_t preload_md5() {
  hipFuncAttributes attr;
  return hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(&md5_prefix_kernel));
}

}  // namespace gleam

extern "C" gleam_status gleam_md5_prefix(const gleam_batch* b, uint32_t prefix_bytes, uint64_t min_len,
                                         uint64_t* d_digest, uint64_t* d_key, uint8_t* d_eligible, void* stream) {
  using namespace gleam;
  clear_error();
  gleam_status st = validate_batch(b, "gleam_md5_prefix");
  if (st != GLEAM_OK) return st;
  if (prefix_bytes > kMaxPrefix) {
    set_error("gleam_md5_prefix: prefix_bytes above %u", kMaxPrefix);
    return GLEAM_E_INVALID;
  }
  if (b->n_seg == 0) return GLEAM_OK;
  if (!b->seg_addr || !b->seg_len || !d_digest) {
    set_error("gleam_md5_prefix: null descriptor or digest output");
    return GLEAM_E_INVALID;
  }
  const uint64_t grid = (b->n_seg + kThreads - 1) / kThreads;
  if (grid > 0x7fffffffull) {
    set_error("gleam_md5_prefix: more than 2^31 workgroups of payloads");
    return GLEAM_E_UNSUPPORTED;
  }
  hipLaunchKernelGGL(md5_prefix_kernel, dim3((uint32_t)grid), dim3(kThreads), 0, (hipStream_t)stream, b->seg_addr,
                     b->seg_len, b->n_seg, prefix_bytes, min_len, d_digest, d_key, d_eligible);
  return launch_status("md5_prefix_kernel");
}
