// Tensor commitments for gfx950: SHA-256 (FIPS 180-4) and the RFC 6962 Merkle
// Tree Hash over fixed-size chunks of a tensor's bytes.
//
// The Verde protocol commits to checkpoints and to the tensors entering and
// leaving every graph node with a collision-resistant hash such as SHA-256,
// and combines node hashes in a binary Merkle tree (Sections 2.1 and 2.2).  A
// single SHA-256 stream is sequential, so a tensor is committed as a Merkle
// tree of its chunks: leaf = SHA-256(0x00 || chunk), node = SHA-256(0x01 ||
// left || right), the tree split at the largest power of two (RFC 6962).
//
// Schedule: one lane per leaf chunk (the chunk's blocks in sequence); then
// the tree level by level, pairs hashed and an odd last node carried up
// unchanged (which reproduces RFC 6962's split): one launch per level while a
// level is wider than 512 nodes, then the rest in one workgroup from LDS, which
// writes the root as 32 bytes.  A level costs at least one two-block hash of
// latency (about 6 us), so a tensor's commitment has a floor of about that
// times the tree depth; wide levels and the leaves are integer-ALU bound.
//
// Digests travel between kernels as eight 32-bit words (SHA-256's big-endian
// word view); data bytes are read as little-endian dwords and reassembled into
// message words with byte permutes, the one-byte prefix shifting every word
// by a byte.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "commit_internal.h"

namespace repops {
namespace {

// First 32 bits of the fractional parts of the cube roots of the first 64
// primes, and of the square roots of the first 8 primes (FIPS 180-4, 4.2.2
// and 5.3.3).
constexpr uint32_t kK[64] = {
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
constexpr uint32_t kH0[8] = {0x6a09e667u, 0xbb67ae85u, 0x3c6ef372u, 0xa54ff53au,
                             0x510e527fu, 0x9b05688cu, 0x1f83d9abu, 0x5be0cd19u};

constexpr int kTopNodes = 512;     // nodes one workgroup reduces to one (nine levels)
constexpr int kTopThreads = 256;

__device__ __forceinline__ uint32_t rotr(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

// SHA-256's three-input bitwise functions, each one gfx950 three-input bitwise
// operation; the 8-bit table holds the output for input bits (a, b, c) at
// bit 4a + 2b + c.  Parity (0x96) for the Sigma / sigma functions, majority
// (0xE8), and choose -- b where a is set, else c -- (0xCA).  (The compiler
// otherwise splits each into two-input operations.)
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}
__device__ __forceinline__ uint32_t maj3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0xE8);
}
__device__ __forceinline__ uint32_t choose(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0xCA);
}

// The compression function on one block; W holds the block's 16 words and is
// consumed as the rolling message schedule.  Fully unrolled: every round
// constant is an immediate.
__device__ __forceinline__ void compress(uint32_t H[8], uint32_t W[16]) {
  uint32_t a = H[0], b = H[1], c = H[2], d = H[3], e = H[4], f = H[5], g = H[6], h = H[7];
#pragma unroll
  for (int t = 0; t < 64; ++t) {
    uint32_t w;
    if (t < 16) {
      w = W[t];
    } else {
      const uint32_t w15 = W[(t - 15) & 15], w2 = W[(t - 2) & 15];
      const uint32_t s0 = xor3(rotr(w15, 7), rotr(w15, 18), w15 >> 3);
      const uint32_t s1 = xor3(rotr(w2, 17), rotr(w2, 19), w2 >> 10);
      w = W[t & 15] + s0 + W[(t - 7) & 15] + s1;
      W[t & 15] = w;
    }
    const uint32_t S1 = xor3(rotr(e, 6), rotr(e, 11), rotr(e, 25));
    const uint32_t ch = choose(e, f, g);
    const uint32_t T1 = h + S1 + ch + kK[t] + w;
    const uint32_t S0 = xor3(rotr(a, 2), rotr(a, 13), rotr(a, 22));
    const uint32_t maj = maj3(a, b, c);
    const uint32_t T2 = S0 + maj;
    h = g;
    g = f;
    f = e;
    e = d + T1;
    d = c;
    c = b;
    b = a;
    a = T1 + T2;
  }
  H[0] += a; H[1] += b; H[2] += c; H[3] += d;
  H[4] += e; H[5] += f; H[6] += g; H[7] += h;
}

// Message word whose bytes are (top byte of prev, bytes 0..2 of cur): the
// stream shifted by the one-byte prefix, with prev/cur little-endian dwords.
__device__ __forceinline__ uint32_t shifted_word(uint32_t prev, uint32_t cur) {
  return (prev & 0xff000000u) | ((cur & 0xffu) << 16) | (cur & 0xff00u) | ((cur >> 16) & 0xffu);
}

// Byte p of (prefix || data[0..len) || 0x80 || zeros || 64-bit bit length),
// padded to `blocks` blocks: the generic path for a short or unaligned chunk.
__device__ __forceinline__ uint32_t stream_byte(const uint8_t* data, uint64_t len, uint8_t prefix,
                                                uint64_t p, uint64_t total_len, uint64_t blocks) {
  if (p == 0) return prefix;
  if (p - 1 < len) return data[p - 1];
  if (p == len + 1) return 0x80u;
  const uint64_t end = blocks * 64;
  if (p >= end - 8) {
    const uint64_t bits = total_len * 8;
    const int shift = static_cast<int>(8 * (end - 1 - p));
    return static_cast<uint32_t>((bits >> shift) & 0xffu);
  }
  return 0u;
}

__device__ void sha_generic(const uint8_t* data, uint64_t len, uint8_t prefix, uint32_t H[8]) {
#pragma unroll
  for (int k = 0; k < 8; ++k) H[k] = kH0[k];
  const uint64_t total = len + 1;
  const uint64_t blocks = (total + 9 + 63) / 64;
  for (uint64_t b = 0; b < blocks; ++b) {
    uint32_t W[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint64_t p = b * 64 + 4 * j;
      W[j] = (stream_byte(data, len, prefix, p, total, blocks) << 24) |
             (stream_byte(data, len, prefix, p + 1, total, blocks) << 16) |
             (stream_byte(data, len, prefix, p + 2, total, blocks) << 8) |
             stream_byte(data, len, prefix, p + 3, total, blocks);
    }
    compress(H, W);
  }
}

// ---------------------------------------------------------------------------
// leaves: H = SHA-256(0x00 || chunk)
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void leaf_kernel(const uint8_t* data, uint64_t nbytes,
                                                   uint32_t chunk, uint64_t leaves, uint32_t* out,
                                                   int vec) {
  const uint64_t leaf = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (leaf >= leaves) return;
  const uint64_t off = leaf * chunk;
  const uint64_t len = (off + chunk <= nbytes) ? chunk : nbytes - off;
  uint32_t H[8];
  if (vec && len == chunk) {
    // Full chunk, 16-byte aligned, chunk a multiple of 64: chunk/64 blocks of
    // (prefix || data), then one block with the last data byte and padding.
#pragma unroll
    for (int k = 0; k < 8; ++k) H[k] = kH0[k];
    const uint4* p = reinterpret_cast<const uint4*>(data + off);
    uint32_t prev = 0;  // the prefix byte 0x00 sits in prev's top byte
    const uint32_t nb = chunk / 64;
    uint4 q0 = p[0], q1 = p[1], q2 = p[2], q3 = p[3];
    for (uint32_t b = 0; b < nb; ++b) {
      const uint32_t d[16] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w,
                              q2.x, q2.y, q2.z, q2.w, q3.x, q3.y, q3.z, q3.w};
      if (b + 1 < nb) {  // next block's loads in flight during this block's rounds
        q0 = p[4 * (b + 1)];
        q1 = p[4 * (b + 1) + 1];
        q2 = p[4 * (b + 1) + 2];
        q3 = p[4 * (b + 1) + 3];
      }
      uint32_t W[16];
      W[0] = shifted_word(prev, d[0]);
#pragma unroll
      for (int j = 1; j < 16; ++j) W[j] = shifted_word(d[j - 1], d[j]);
      prev = d[15];
      compress(H, W);
    }
    const uint64_t bits = (static_cast<uint64_t>(chunk) + 1) * 8;
    uint32_t W[16];
    W[0] = (prev & 0xff000000u) | 0x00800000u;
#pragma unroll
    for (int j = 1; j < 14; ++j) W[j] = 0;
    W[14] = static_cast<uint32_t>(bits >> 32);
    W[15] = static_cast<uint32_t>(bits);
    compress(H, W);
  } else {
    sha_generic(data + off, len, 0x00, H);
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) out[leaf * 8 + k] = H[k];
}

// ---------------------------------------------------------------------------
// nodes: H = SHA-256(0x01 || L || R), 65 bytes = two blocks
// ---------------------------------------------------------------------------

__device__ __forceinline__ void node_hash(const uint32_t L[8], const uint32_t R[8], uint32_t H[8]) {
#pragma unroll
  for (int k = 0; k < 8; ++k) H[k] = kH0[k];
  uint32_t W[16];
  W[0] = 0x01000000u | (L[0] >> 8);
#pragma unroll
  for (int j = 1; j < 8; ++j) W[j] = (L[j - 1] << 24) | (L[j] >> 8);
  W[8] = (L[7] << 24) | (R[0] >> 8);
#pragma unroll
  for (int j = 9; j < 16; ++j) W[j] = (R[j - 9] << 24) | (R[j - 8] >> 8);
  compress(H, W);
  W[0] = (R[7] << 24) | 0x00800000u;
#pragma unroll
  for (int j = 1; j < 15; ++j) W[j] = 0;
  W[15] = 65 * 8;
  compress(H, W);
}

__global__ __launch_bounds__(256) void node_kernel(const uint32_t* in, uint64_t n_in,
                                                   uint32_t* out) {
  const uint64_t i = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const uint64_t n_out = (n_in + 1) / 2;
  if (i >= n_out) return;
  uint32_t H[8];
  if (2 * i + 1 < n_in) {
    uint32_t L[8], R[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      L[k] = in[(2 * i) * 8 + k];
      R[k] = in[(2 * i + 1) * 8 + k];
    }
    node_hash(L, R, H);
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) H[k] = in[(2 * i) * 8 + k];  // odd last node carried up
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) out[i * 8 + k] = H[k];
}

// The last levels (at most kTopNodes nodes) in one workgroup, level by level
// in LDS; the root is written as 32 bytes in SHA-256's byte order.  (The
// kernel also reduces aligned slices of kTopNodes nodes when launched with
// several workgroups -- inside such a slice the pairs (2i, 2i + 1) are those
// of the whole level and only the last slice can hold the odd last node -- but
// wide levels run faster one launch per level: inside a workgroup every level
// after the first leaves half of the remaining lanes idle, while a level costs
// about one two-block hash of latency either way.)
__global__ __launch_bounds__(kTopThreads) void tree_kernel(const uint32_t* in, uint64_t n_in,
                                                           uint32_t* out, uint8_t* digest) {
  __shared__ uint32_t buf[2][kTopNodes * 8];
  const int tid = threadIdx.x;
  const uint64_t first = static_cast<uint64_t>(blockIdx.x) * kTopNodes;
  const uint64_t left = n_in - first;
  uint64_t n = left < static_cast<uint64_t>(kTopNodes) ? left : kTopNodes;
  for (uint64_t i = tid; i < n * 8; i += kTopThreads) buf[0][i] = in[first * 8 + i];
  __syncthreads();
  int cur = 0;
  while (n > 1) {
    const uint64_t n_out = (n + 1) / 2;
    for (uint64_t i = tid; i < n_out; i += kTopThreads) {
      uint32_t H[8];
      if (2 * i + 1 < n) {
        uint32_t L[8], R[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          L[k] = buf[cur][(2 * i) * 8 + k];
          R[k] = buf[cur][(2 * i + 1) * 8 + k];
        }
        node_hash(L, R, H);
      } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) H[k] = buf[cur][(2 * i) * 8 + k];
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) buf[cur ^ 1][i * 8 + k] = H[k];
    }
    __syncthreads();
    cur ^= 1;
    n = n_out;
  }
  if (digest) {
    if (tid < 32) {
      const uint32_t w = buf[cur][tid / 4];
      digest[tid] = static_cast<uint8_t>(w >> (24 - 8 * (tid % 4)));
    }
  } else if (tid < 8) {
    out[static_cast<uint64_t>(blockIdx.x) * 8 + tid] = buf[cur][tid];
  }
}

// SHA-256 of the empty message (the commitment of zero bytes).
__global__ __launch_bounds__(64) void empty_kernel(uint8_t* digest) {
  uint32_t H[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) H[k] = kH0[k];
  uint32_t W[16];
  W[0] = 0x80000000u;
#pragma unroll
  for (int j = 1; j < 16; ++j) W[j] = 0;
  compress(H, W);
  const int tid = threadIdx.x;
  if (tid < 32) digest[tid] = static_cast<uint8_t>(H[tid / 4] >> (24 - 8 * (tid % 4)));
}

unsigned grid_for(uint64_t items, int threads) {
  return static_cast<unsigned>((items + threads - 1) / threads);
}

}  // namespace

uint64_t commit_leaves(uint64_t nbytes, uint32_t chunk) {
  return nbytes == 0 ? 0 : (nbytes + chunk - 1) / chunk;
}

uint64_t commit_workspace_bytes(uint64_t nbytes, uint32_t chunk) {
  const uint64_t leaves = commit_leaves(nbytes, chunk);
  return 32 * (leaves + (leaves + 1) / 2);
}

hipError_t launch_commit(const uint8_t* data, uint64_t nbytes, uint32_t chunk, uint8_t* digest,
                         uint32_t* ws, hipStream_t s) {
  const uint64_t leaves = commit_leaves(nbytes, chunk);
  if (leaves == 0) {
    hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, s, digest);
    return hipGetLastError();
  }
  const bool vec = reinterpret_cast<uintptr_t>(data) % 16 == 0 && chunk % 64 == 0;
  uint32_t* a = ws;                // leaf digests, then every second reduced level
  uint32_t* b = ws + leaves * 8;   // the other reduced levels
  hipLaunchKernelGGL(leaf_kernel, dim3(grid_for(leaves, 256)), dim3(256), 0, s, data, nbytes,
                     chunk, leaves, a, vec ? 1 : 0);
  hipError_t e = hipGetLastError();
  uint64_t n = leaves;
  while (e == hipSuccess && n > static_cast<uint64_t>(kTopNodes)) {
    hipLaunchKernelGGL(node_kernel, dim3(grid_for((n + 1) / 2, 256)), dim3(256), 0, s, a, n, b);
    e = hipGetLastError();
    uint32_t* t = a;
    a = b;
    b = t;
    n = (n + 1) / 2;
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(tree_kernel, dim3(1), dim3(kTopThreads), 0, s, a, n,
                     static_cast<uint32_t*>(nullptr), digest);
  return hipGetLastError();
}

}  // namespace repops
