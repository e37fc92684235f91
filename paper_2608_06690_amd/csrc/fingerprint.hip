// Weight fingerprint: a 16-ary SHA-256 tree over a device buffer.
//
// The frozen public weights are hashed before and after training and after a reload, and
// the digests must agree (Sec. 3.2 training and checkpointing; Sec. 5.1; App. C.1).
// The tree lets every level run in parallel: level 0 hashes each 1 KiB chunk of the
// buffer, every higher level hashes each run of up to 16 consecutive digests of the level
// below, until one digest is left. An input of at most 1 KiB therefore has the plain
// SHA-256 of its bytes as its fingerprint.
//
// SHA-256 follows FIPS 180-4: message padding (5.1.1), initial hash value (5.3.3),
// round constants (4.2.2), message schedule and compression (6.2.2). Words are
// big-endian, so bytes are swapped on load and on store; the stored digest bytes are
// the standard digest.
//
// One thread hashes one chunk; a chunk is processed 64 bytes at a time. SHA-256 is
// bound by integer VALU work (about 23 operations per input byte), not by HBM.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

// FIPS 180-4 4.2.2: first 32 bits of the fractional parts of the cube roots of the
// first 64 primes.
constexpr uint32_t kRound[64] = {
    0x428a2f98u, 0x71374491u, 0xb5c0fbcfu, 0xe9b5dba5u, 0x3956c25bu, 0x59f111f1u, 0x923f82a4u,
    0xab1c5ed5u, 0xd807aa98u, 0x12835b01u, 0x243185beu, 0x550c7dc3u, 0x72be5d74u, 0x80deb1feu,
    0x9bdc06a7u, 0xc19bf174u, 0xe49b69c1u, 0xefbe4786u, 0x0fc19dc6u, 0x240ca1ccu, 0x2de92c6fu,
    0x4a7484aau, 0x5cb0a9dcu, 0x76f988dau, 0x983e5152u, 0xa831c66du, 0xb00327c8u, 0xbf597fc7u,
    0xc6e00bf3u, 0xd5a79147u, 0x06ca6351u, 0x14292967u, 0x27b70a85u, 0x2e1b2138u, 0x4d2c6dfcu,
    0x53380d13u, 0x650a7354u, 0x766a0abbu, 0x81c2c92eu, 0x92722c85u, 0xa2bfe8a1u, 0xa81a664bu,
    0xc24b8b70u, 0xc76c51a3u, 0xd192e819u, 0xd6990624u, 0xf40e3585u, 0x106aa070u, 0x19a4c116u,
    0x1e376c08u, 0x2748774cu, 0x34b0bcb5u, 0x391c0cb3u, 0x4ed8aa4au, 0x5b9cca4fu, 0x682e6ff3u,
    0x748f82eeu, 0x78a5636fu, 0x84c87814u, 0x8cc70208u, 0x90befffau, 0xa4506cebu, 0xbef9a3f7u,
    0xc67178f2u};

// FIPS 180-4 5.3.3: first 32 bits of the fractional parts of the square roots of the
// first 8 primes.
constexpr uint32_t kInit[8] = {0x6a09e667u, 0xbb67ae85u, 0x3c6ef372u, 0xa54ff53au,
                                  0x510e527fu, 0x9b05688cu, 0x1f83d9abu, 0x5be0cd19u};

__device__ __forceinline__ uint32_t rotr(uint32_t x, int n) { return __builtin_rotateright32(x, n); }

// a ^ b ^ c in one CDNA4 three-input bitwise operation (truth table 0x96 = odd parity)
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

// One compression (FIPS 180-4 6.2.2) of the 16-word block w into state s. The message
// schedule is kept as a rolling window of 16 words in w itself (w is overwritten).
__device__ __forceinline__ void compress(uint32_t (&s)[8], uint32_t (&w)[16]) {
  uint32_t a = s[0], b = s[1], c = s[2], d = s[3], e = s[4], f = s[5], g = s[6], h = s[7];
#pragma unroll
  for (int t = 0; t < 64; ++t) {
    uint32_t wt;
    if (t < 16) {
      wt = w[t];
    } else {
      const uint32_t w15 = w[(t - 15) & 15], w2 = w[(t - 2) & 15];
      const uint32_t s0 = xor3(rotr(w15, 7), rotr(w15, 18), w15 >> 3);
      const uint32_t s1 = xor3(rotr(w2, 17), rotr(w2, 19), w2 >> 10);
      wt = w[t & 15] + s0 + w[(t - 7) & 15] + s1;
      w[t & 15] = wt;
    }
    const uint32_t S1 = xor3(rotr(e, 6), rotr(e, 11), rotr(e, 25));
    const uint32_t ch = (e & f) ^ (~e & g);
    const uint32_t t1 = h + S1 + ch + kRound[t] + wt;
    const uint32_t S0 = xor3(rotr(a, 2), rotr(a, 13), rotr(a, 22));
    const uint32_t maj = (a & b) ^ (a & c) ^ (b & c);
    const uint32_t t2 = S0 + maj;
    h = g;
    g = f;
    f = e;
    e = d + t1;
    d = c;
    c = b;
    b = a;
    a = t1 + t2;
  }
  s[0] += a; s[1] += b; s[2] += c; s[3] += d;
  s[4] += e; s[5] += f; s[6] += g; s[7] += h;
}

// Thread c hashes bytes [c*chunk, min((c+1)*chunk, nbytes)) of src into out[32c, 32c+32).
// kAligned: src and chunk are 16-byte aligned, so whole blocks load as four uint4.
template <bool kAligned>
__global__ __launch_bounds__(64) void sha256_chunks_kernel(const uint8_t* __restrict__ src,
                                                           uint64_t nbytes, uint32_t chunk,
                                                           uint64_t nchunks,
                                                           uint8_t* __restrict__ out) {
  const uint64_t c = (uint64_t)blockIdx.x * 64 + threadIdx.x;
  if (c >= nchunks) return;
  const uint64_t off = c * chunk;
  const uint32_t len = (uint32_t)(nbytes - off < chunk ? nbytes - off : chunk);
  const uint8_t* p = src + off;

  uint32_t s[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) s[i] = kInit[i];

  uint32_t w[16];
  const uint32_t nfull = len >> 6;
  for (uint32_t blk = 0; blk < nfull; ++blk, p += 64) {
    if (kAligned) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(p + 16 * q);
        w[4 * q + 0] = __builtin_bswap32(v.x);
        w[4 * q + 1] = __builtin_bswap32(v.y);
        w[4 * q + 2] = __builtin_bswap32(v.z);
        w[4 * q + 3] = __builtin_bswap32(v.w);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i)
        w[i] = ((uint32_t)p[4 * i] << 24) | ((uint32_t)p[4 * i + 1] << 16) |
               ((uint32_t)p[4 * i + 2] << 8) | (uint32_t)p[4 * i + 3];
    }
    compress(s, w);
  }

  // Padding (FIPS 180-4 5.1.1): the r = len mod 64 remaining bytes, one 0x80 byte, zeros,
  // then the message length in bits as a 64-bit big-endian integer in the last 8 bytes;
  // when r >= 56 the length spills into a second block.
  const uint32_t r = len & 63u;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    uint32_t word = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t j = 4 * i + k;
      const uint32_t byte = j < r ? (uint32_t)p[j] : (j == r ? 0x80u : 0u);
      word |= byte << (24 - 8 * k);
    }
    w[i] = word;
  }
  const uint64_t bits = (uint64_t)len * 8;
  if (r >= 56) {
    compress(s, w);
#pragma unroll
    for (int i = 0; i < 14; ++i) w[i] = 0;
  }
  w[14] = (uint32_t)(bits >> 32);
  w[15] = (uint32_t)bits;
  compress(s, w);

  u32x4* o = reinterpret_cast<u32x4*>(out + 32 * c);
  o[0] = u32x4{__builtin_bswap32(s[0]), __builtin_bswap32(s[1]), __builtin_bswap32(s[2]),
               __builtin_bswap32(s[3])};
  o[1] = u32x4{__builtin_bswap32(s[4]), __builtin_bswap32(s[5]), __builtin_bswap32(s[6]),
               __builtin_bswap32(s[7])};
}

hipError_t launch_level(const uint8_t* src, uint64_t nbytes, uint32_t chunk, uint64_t nchunks,
                        uint8_t* out, bool aligned, hipStream_t stream) {
  const dim3 grid((unsigned)((nchunks + 63) / 64));
  if (aligned)
    sha256_chunks_kernel<true><<<grid, 64, 0, stream>>>(src, nbytes, chunk, nchunks, out);
  else
    sha256_chunks_kernel<false><<<grid, 64, 0, stream>>>(src, nbytes, chunk, nchunks, out);
  return hipGetLastError();
}

}  // namespace

uint64_t fingerprint_leaves(uint64_t nbytes) {
  const uint64_t n = (nbytes + kFpLeafBytes - 1) / kFpLeafBytes;
  return n == 0 ? 1 : n;
}

hipError_t launch_fingerprint(const FingerprintArgs& a, hipStream_t stream) {
  uint64_t n = fingerprint_leaves(a.nbytes);
  const bool aligned = ((uintptr_t)a.data & 15u) == 0;
  uint8_t* buf[2] = {a.ws, a.ws2};
  int cur = 0;
  hipError_t e = launch_level((const uint8_t*)a.data, a.nbytes, kFpLeafBytes, n,
                              n == 1 ? a.digest : buf[cur], aligned, stream);
  while (e == hipSuccess && n > 1) {
    const uint64_t m = (n + kFpFanout - 1) / kFpFanout;
    e = launch_level(buf[cur], n * 32, kFpFanout * 32, m, m == 1 ? a.digest : buf[cur ^ 1], true,
                     stream);
    cur ^= 1;
    n = m;
  }
  return e;
}

}  // namespace pmpe
