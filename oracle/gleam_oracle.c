/*
 * Reference oracle for weight-cache hit detection: fingerprints.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the plain, slow, obviously correct CPU
 * definition that the GPU library is checked against. Only the test suite, the
 * package smoke check and the benchmark's CPU-baseline leg load it. The GPU
 * library shares no code, header, table or constant with it, and never calls it.
 *
 * What it computes (Gleam, Sec. 4.1.2 "Hash-based Weight Chunk Retrieval"):
 * every host-to-device copy payload gets a hash identifier computed from its
 * source bytes, and the identifier decides whether the bytes must cross the
 * network. Here the identifier is taken per fixed-size block of each payload:
 *
 *   - geometry: a payload of len bytes is cut, from its first byte, into
 *     leaves of leaf_bytes and blocks of block_bytes (a whole number of
 *     leaves); the last leaf and the last block may be partial and are hashed
 *     over their actual bytes, without padding;
 *   - leaf digest: XXH64 with seed 0 over the leaf's bytes (the 64-bit xxHash
 *     algorithm as published in the xxHash specification by Y. Collet);
 *   - block digest: a bottom-up pairwise tree over the block's leaf digests;
 *     a node is XXH64(LE64(left) || LE64(right), seed 0), and an odd element
 *     at the end of a level moves up unchanged. One leaf: the leaf digest.
 *
 * Nothing here is blocked, fused or reordered: one scalar pass per leaf, one
 * level of the tree at a time.
 *
 * It also holds MD5 (RFC 1321) for the paper's own identifier (see oracle_md5).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* The five 64-bit primes of the XXH64 specification. */
#define XP1 0x9E3779B185EBCA87ULL
#define XP2 0xC2B2AE3D27D4EB4FULL
#define XP3 0x165667B19E3779F9ULL
#define XP4 0x85EBCA77C2B2AE63ULL
#define XP5 0x27D4EB2F165667C5ULL

static uint64_t rotate_left(uint64_t x, unsigned r) { return (x << r) | (x >> (64u - r)); }

/* Little-endian reads, byte by byte, so the result does not depend on the host. */
static uint64_t read_le64(const uint8_t* p) {
  uint64_t v = 0;
  for (int i = 7; i >= 0; --i) v = (v << 8) | p[i];
  return v;
}
static uint32_t read_le32(const uint8_t* p) {
  uint32_t v = 0;
  for (int i = 3; i >= 0; --i) v = (v << 8) | p[i];
  return v;
}

/* One accumulator step of the specification: acc <- rotl(acc + lane*P2, 31) * P1. */
static uint64_t xxh64_round(uint64_t acc, uint64_t lane) {
  acc += lane * XP2;
  acc = rotate_left(acc, 31);
  return acc * XP1;
}

/* Folding an accumulator into the hash after the stripe loop. */
static uint64_t xxh64_merge(uint64_t h, uint64_t acc) {
  h ^= xxh64_round(0, acc);
  return h * XP1 + XP4;
}

uint64_t oracle_xxh64(const uint8_t* p, uint64_t len, uint64_t seed) {
  uint64_t h;
  uint64_t pos = 0;
  if (len >= 32) {
    uint64_t v1 = seed + XP1 + XP2;
    uint64_t v2 = seed + XP2;
    uint64_t v3 = seed;
    uint64_t v4 = seed - XP1;
    /* every whole 32-byte stripe: four 8-byte lanes, one per accumulator */
    while (pos + 32 <= len) {
      v1 = xxh64_round(v1, read_le64(p + pos + 0));
      v2 = xxh64_round(v2, read_le64(p + pos + 8));
      v3 = xxh64_round(v3, read_le64(p + pos + 16));
      v4 = xxh64_round(v4, read_le64(p + pos + 24));
      pos += 32;
    }
    h = rotate_left(v1, 1) + rotate_left(v2, 7) + rotate_left(v3, 12) + rotate_left(v4, 18);
    h = xxh64_merge(h, v1);
    h = xxh64_merge(h, v2);
    h = xxh64_merge(h, v3);
    h = xxh64_merge(h, v4);
  } else {
    h = seed + XP5;
  }
  h += len;
  /* the remaining bytes: 8 at a time, then 4, then one by one */
  while (pos + 8 <= len) {
    h ^= xxh64_round(0, read_le64(p + pos));
    h = rotate_left(h, 27) * XP1 + XP4;
    pos += 8;
  }
  if (pos + 4 <= len) {
    h ^= (uint64_t)read_le32(p + pos) * XP1;
    h = rotate_left(h, 23) * XP2 + XP3;
    pos += 4;
  }
  while (pos < len) {
    h ^= (uint64_t)p[pos] * XP5;
    h = rotate_left(h, 11) * XP1;
    pos += 1;
  }
  /* final avalanche */
  h ^= h >> 33;
  h *= XP2;
  h ^= h >> 29;
  h *= XP3;
  h ^= h >> 32;
  return h;
}

/* Tree node: the digest of the 16-byte string LE64(left) || LE64(right). */
uint64_t oracle_node(uint64_t left, uint64_t right) {
  uint8_t buf[16];
  for (int i = 0; i < 8; ++i) {
    buf[i] = (uint8_t)(left >> (8 * i));
    buf[8 + i] = (uint8_t)(right >> (8 * i));
  }
  return oracle_xxh64(buf, 16, 0);
}

/* Bottom-up tree over n >= 1 digests; `work` is overwritten. */
uint64_t oracle_tree(uint64_t* work, uint64_t n) {
  while (n > 1) {
    uint64_t m = 0;
    for (uint64_t i = 0; i + 1 < n; i += 2) work[m++] = oracle_node(work[i], work[i + 1]);
    if (n % 2 == 1) work[m++] = work[n - 1]; /* odd element moves up unchanged */
    n = m;
  }
  return work[0];
}

uint64_t oracle_num_blocks(uint64_t len, uint32_t block_bytes) {
  return (len + block_bytes - 1) / block_bytes;
}

/*
 * Digests of blocks [first_block, first_block + count) of one payload.
 *   payload, len      : the payload's bytes (host memory) and length
 *   leaf_bytes        : leaf size (4096 in every workload here)
 *   block_bytes       : block size, a whole multiple of leaf_bytes
 *   block_out[count]  : block digests
 *   leaf_out          : NULL, or [count * (block_bytes / leaf_bytes)] leaf
 *                       digests, block-major; slots past a partial block's
 *                       last leaf are set to 0
 * Returns 0 on success, -1 on an invalid argument, -2 if memory ran out.
 */
int oracle_blocks(const uint8_t* payload, uint64_t len, uint32_t leaf_bytes, uint32_t block_bytes,
                  uint64_t first_block, uint64_t count, uint64_t* block_out, uint64_t* leaf_out) {
  if (leaf_bytes == 0 || block_bytes == 0 || block_bytes % leaf_bytes != 0) return -1;
  uint64_t nblk = oracle_num_blocks(len, block_bytes);
  if (first_block + count > nblk) return -1;
  uint64_t per_block = block_bytes / leaf_bytes;
  uint64_t* work = (uint64_t*)malloc(per_block * sizeof(uint64_t));
  if (!work) return -2;
  for (uint64_t b = 0; b < count; ++b) {
    uint64_t j = first_block + b;
    uint64_t start = j * (uint64_t)block_bytes;
    uint64_t end = start + block_bytes;
    if (end > len) end = len;
    uint64_t nleaf = 0;
    for (uint64_t off = start; off < end; off += leaf_bytes) {
      uint64_t leaf_end = off + leaf_bytes;
      if (leaf_end > end) leaf_end = end;
      work[nleaf++] = oracle_xxh64(payload + off, leaf_end - off, 0);
    }
    if (leaf_out) {
      for (uint64_t k = 0; k < per_block; ++k) leaf_out[b * per_block + k] = k < nleaf ? work[k] : 0;
    }
    block_out[b] = oracle_tree(work, nleaf);
  }
  free(work);
  return 0;
}

/*
 * MD5 (RFC 1321), used for the paper's own identifier (Appendix, discussion of hash
 * cost and collisions: an MD5 string of the first 1024 bits of each host-to-device
 * chunk). Written from the RFC's description: the message is padded with one 1 bit,
 * zeros to 56 mod 64 bytes and the 64-bit little-endian bit length; each 64-byte block
 * runs four rounds of sixteen steps a = b + ((a + fn(b,c,d) + X[k] + T[i]) <<< s)
 * over the state A, B, C, D. T[i] is the integer part of 2^32 * |sin(i)| (i in radians),
 * computed here from that definition.
 */

static uint32_t md5_rotl(uint32_t x, unsigned s) { return (x << s) | (x >> (32u - s)); }

static void md5_block(uint32_t state[4], const uint8_t block[64], const uint32_t T[65]) {
  static const unsigned S[4][4] = {{7, 12, 17, 22}, {5, 9, 14, 20}, {4, 11, 16, 23}, {6, 10, 15, 21}};
  uint32_t X[16];
  for (int j = 0; j < 16; ++j) X[j] = read_le32(block + 4 * j);
  uint32_t a = state[0], b = state[1], c = state[2], d = state[3];
  for (int i = 0; i < 64; ++i) {
    const int round = i / 16;
    uint32_t f;
    int k;
    if (round == 0) {        /* F(X,Y,Z) = XY v not(X) Z */
      f = (b & c) | (~b & d);
      k = i;
    } else if (round == 1) { /* G(X,Y,Z) = XZ v Y not(Z) */
      f = (b & d) | (c & ~d);
      k = (5 * i + 1) % 16;
    } else if (round == 2) { /* H(X,Y,Z) = X xor Y xor Z */
      f = b ^ c ^ d;
      k = (3 * i + 5) % 16;
    } else {                 /* I(X,Y,Z) = Y xor (X v not(Z)) */
      f = c ^ (b | ~d);
      k = (7 * i) % 16;
    }
    const uint32_t t = a + f + X[k] + T[i + 1];
    a = d;
    d = c;
    c = b;
    b = b + md5_rotl(t, S[round][i % 4]);
  }
  state[0] += a;
  state[1] += b;
  state[2] += c;
  state[3] += d;
}

/* MD5 of p[0..len); out receives the 16-byte digest (A, B, C, D little-endian). */
void oracle_md5(const uint8_t* p, uint64_t len, uint8_t out[16]) {
  uint32_t T[65];
  for (int i = 1; i <= 64; ++i) T[i] = (uint32_t)floor(4294967296.0 * fabs(sin((double)i)));
  uint32_t state[4] = {0x67452301u, 0xefcdab89u, 0x98badcfeu, 0x10325476u};
  uint64_t pos = 0;
  for (; pos + 64 <= len; pos += 64) md5_block(state, p + pos, T);
  uint8_t tail[128];
  const uint64_t rem = len - pos;
  memset(tail, 0, sizeof tail);
  if (rem) memcpy(tail, p + pos, rem);
  tail[rem] = 0x80;
  const uint64_t tail_len = rem + 1 + 8 <= 64 ? 64 : 128;
  const uint64_t bits = len * 8;
  for (int i = 0; i < 8; ++i) tail[tail_len - 8 + i] = (uint8_t)(bits >> (8 * i));
  md5_block(state, tail, T);
  if (tail_len == 128) md5_block(state, tail + 64, T);
  for (int w = 0; w < 4; ++w)
    for (int i = 0; i < 4; ++i) out[4 * w + i] = (uint8_t)(state[w] >> (8 * i));
}
