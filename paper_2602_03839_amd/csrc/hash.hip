// hash.hip -- the weight-level integrity hash of App. J.4 on gfx950.
//
// The paper hashes the BF16 bit patterns of all parameters, concatenated in a
// fixed order, with SHA-256, so that a receiver can check the weights it
// rebuilt from a patch chain.  One SHA-256 over the whole stream is a single
// chain of compressions that no GPU can split, so the hash is a tree of
// SHA-256: the stream (each value's two bytes, low byte first) is cut into
// 16 KiB leaves and combined with the Merkle Tree Hash of RFC 6962, Sec. 2.1
// (leaf = SHA-256(0x00 || chunk), node = SHA-256(0x01 || left || right), the
// left subtree holding the largest power of two of leaves below the count).
//
// SHA-256 (FIPS 180-4) is 32-bit integer work: about 1,650 VALU operations per
// 64-byte block, ~26 per byte, so the kernel is bound by the vector ALU, not
// by HBM (it reads 2 bytes per parameter once).  One lane hashes one leaf;
// lanes of a wave hash neighbouring leaves, 16 KiB apart, and each lane reads
// its own 64-byte blocks with 16-byte loads.
//
// Kernels:
//   hash_setup_kernel  writes the tensor table and gathers the leaves that
//                      cross a tensor boundary into scratch slots;
//   hash_leaf_kernel   one lane per leaf: its digest;
//   hash_tree_kernel   one block per 512 digests: the 9 tree levels above
//                      them, in LDS; the host repeats it until one remains.
#include "launch.hpp"

namespace pulse {
namespace {

// ---------------------------------------------------------------------------
// FIPS 180-4 constants from their definitions (5.3.3, 4.2.2): the first 32
// bits of the fractional parts of the square roots of the first 8 primes and
// of the cube roots of the first 64 primes, as integer Newton roots evaluated
// by the compiler.
constexpr uint64_t newton_root(unsigned __int128 v, int e) {
  unsigned __int128 y = (unsigned __int128)1 << 40;  // above every root taken here
  for (;;) {
    unsigned __int128 z = e == 2 ? (y + v / y) / 2 : (2 * y + v / (y * y)) / 3;
    if (z >= y) return (uint64_t)y;
    y = z;
  }
}

struct ShaConsts {
  uint32_t k[64];
  uint32_t h0[8];
};

constexpr ShaConsts make_sha_consts() {
  ShaConsts c{};
  int found = 0;
  for (uint64_t p = 2; found < 64; ++p) {
    bool prime = true;
    for (uint64_t d = 2; d * d <= p; ++d)
      if (p % d == 0) prime = false;
    if (!prime) continue;
    c.k[found] = (uint32_t)newton_root((unsigned __int128)p << 96, 3);
    if (found < 8) c.h0[found] = (uint32_t)newton_root((unsigned __int128)p << 64, 2);
    ++found;
  }
  return c;
}

constexpr ShaConsts kSha = make_sha_consts();
static_assert(kSha.h0[0] == 0x6a09e667u && kSha.k[0] == 0x428a2f98u && kSha.k[63] == 0xc67178f2u,
              "SHA-256 constants");

__device__ __forceinline__ uint32_t rotr(uint32_t x, int n) {
  return __builtin_amdgcn_alignbit(x, x, n);
}

// gfx950's three-input bitwise instruction: the 8-bit immediate is the truth
// table, indexed by (x << 2) | (y << 1) | z over the operand bits.
__device__ __forceinline__ uint32_t xor3(uint32_t x, uint32_t y, uint32_t z) {
  return __builtin_amdgcn_bitop3_b32(x, y, z, 0x96);
}
__device__ __forceinline__ uint32_t ch(uint32_t x, uint32_t y, uint32_t z) {  // x ? y : z
  return __builtin_amdgcn_bitop3_b32(x, y, z, 0xCA);
}
__device__ __forceinline__ uint32_t maj(uint32_t x, uint32_t y, uint32_t z) {  // majority
  return __builtin_amdgcn_bitop3_b32(x, y, z, 0xE8);
}

// One SHA-256 compression (FIPS 180-4, 6.2.2) of the 16 message words w into st.
__device__ __forceinline__ void sha256_block(uint32_t (&st)[8], uint32_t (&w)[16]) {
  uint32_t a = st[0], b = st[1], c = st[2], d = st[3];
  uint32_t e = st[4], f = st[5], g = st[6], h = st[7];
#pragma unroll
  for (int t = 0; t < 64; ++t) {
    uint32_t wt;
    if (t < 16) {
      wt = w[t];
    } else {
      const uint32_t x = w[(t - 15) & 15], y = w[(t - 2) & 15];
      const uint32_t s0 = xor3(rotr(x, 7), rotr(x, 18), x >> 3);
      const uint32_t s1 = xor3(rotr(y, 17), rotr(y, 19), y >> 10);
      wt = w[t & 15] + s0 + w[(t - 7) & 15] + s1;
      w[t & 15] = wt;
    }
    const uint32_t S1 = xor3(rotr(e, 6), rotr(e, 11), rotr(e, 25));
    const uint32_t t1 = h + S1 + ch(e, f, g) + kSha.k[t] + wt;
    const uint32_t S0 = xor3(rotr(a, 2), rotr(a, 13), rotr(a, 22));
    const uint32_t t2 = S0 + maj(a, b, c);
    h = g;
    g = f;
    f = e;
    e = d + t1;
    d = c;
    c = b;
    b = a;
    a = t1 + t2;
  }
  st[0] += a;
  st[1] += b;
  st[2] += c;
  st[3] += d;
  st[4] += e;
  st[5] += f;
  st[6] += g;
  st[7] += h;
}

__device__ __forceinline__ void sha256_init(uint32_t (&st)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) st[i] = kSha.h0[i];
}

typedef uint32_t u32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));
typedef const __attribute__((address_space(1))) u32x4_a4* gvec;  // global memory
typedef const __attribute__((address_space(1))) uint32_t* gword;

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void hash_setup_kernel(HashSetupParams p) {
  if (blockIdx.x == 0 && threadIdx.x < p.nentries)
    p.table[p.first_entry + threadIdx.x] = p.entries[threadIdx.x];
  if (blockIdx.x >= p.njobs) return;
  const HashCopyJob j = p.jobs[blockIdx.x];
  uint16_t* dst = (uint16_t*)(p.scratch + j.dst);
  for (uint64_t i = threadIdx.x; i < j.count; i += blockDim.x) dst[i] = j.src[i];
}

// ---------------------------------------------------------------------------
// Leaf digests.  Message of leaf l: 0x00 followed by its len bytes.  Message
// word k (big-endian, FIPS 180-4 5.2.1) is the 4 bytes at message offset 4k,
// i.e. stream bytes 4k-1 .. 4k+2 of the leaf: the high byte of one 4-byte
// word of the source and three bytes of the next, put in order by one
// v_perm_b32.  A leaf whose source starts 2 bytes into a word (after a tensor
// of odd length) takes the other byte selector.
__global__ __launch_bounds__(256) void hash_leaf_kernel(HashLeafParams p) {
  const uint64_t l = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (l >= p.nleaves) return;
  const uint64_t x = l * kHashLeafElems;
  const uint64_t le = p.total - x < kHashLeafElems ? p.total - x : kHashLeafElems;
  const uint32_t len = (uint32_t)(2 * le);

  uint32_t lo = 0, hi = p.ntensors;
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (p.table[mid].off <= x) lo = mid;
    else hi = mid;
  }
  const HashEntry t = p.table[lo];
  const uint64_t end = p.table[lo + 1].off;

  // Source words: base[0 .. dmax] hold the leaf's bytes, starting sh bytes
  // into base[0]; message word k pairs base[k - 1 + o] with base[k + o].
  const uint32_t* base;
  uint32_t sel, prev, o, dmax;
  if (hash_leaf_in_place(x, le, t.off, end)) {
    const uintptr_t A = (uintptr_t)(t.ptr + (x - t.off));
    const uint32_t sh = (uint32_t)(A & 3);  // 0 or 2
    base = (const uint32_t*)(A - sh);
    o = sh >> 1;
    prev = sh ? (base[0] & 0xFFFF0000u) : 0u;  // the bytes before the leaf read as the prefix 0
    sel = sh ? 0x05060700u : 0x07000102u;
    dmax = (sh + len + 3) / 4 - 1;
  } else {
    base = (const uint32_t*)(p.scratch + (uint64_t)lo * kHashLeafBytes);
    o = 0;
    prev = 0u;
    sel = 0x07000102u;
    dmax = (len + 3) / 4 - 1;
  }

  uint32_t st[8];
  sha256_init(st);
  const uint32_t nfull = (len + 1) / 64;  // blocks made of message bytes only
  for (uint32_t b = 0; b < nfull; ++b) {
    const gvec q = (gvec)(base + 16 * b + o);
    uint32_t d[16];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const u32x4_a4 v = __builtin_nontemporal_load(q + i);
      d[4 * i] = v.x;
      d[4 * i + 1] = v.y;
      d[4 * i + 2] = v.z;
      d[4 * i + 3] = v.w;
    }
    uint32_t w[16];
    w[0] = __builtin_amdgcn_perm(prev, d[0], sel);
#pragma unroll
    for (int j = 1; j < 16; ++j) w[j] = __builtin_amdgcn_perm(d[j - 1], d[j], sel);
    prev = d[15];
    sha256_block(st, w);
  }
  // The last one or two blocks: the message's tail, the byte 0x80, zeros and
  // the bit length (FIPS 180-4 5.1.1).  Reads are clamped to base[dmax]; the
  // bytes past the message that such a read brings in are masked off.
  const uint32_t nblocks = (len + 1 + 1 + 8 + 63) / 64;
  for (uint32_t b = nfull; b < nblocks; ++b) {
    uint32_t w[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t k = 16 * b + j;
      const uint32_t cur = ((gword)base)[k + o < dmax ? k + o : dmax];
      uint32_t word = __builtin_amdgcn_perm(prev, cur, sel);
      prev = cur;
      const int nb = (int)(len + 1) - (int)(4 * k);  // message bytes left at this word
      word &= nb >= 4 ? 0xFFFFFFFFu : nb <= 0 ? 0u : ~(0xFFFFFFFFu >> (8 * nb));
      if (nb >= 0 && nb < 4) word |= 0x80u << (24 - 8 * nb);
      w[j] = word;
    }
    if (b == nblocks - 1) {
      w[14] = 0;
      w[15] = 8 * (len + 1);
    }
    sha256_block(st, w);
  }

  uint32_t* out = (uint32_t*)(p.digests + 32 * l);
  u32x4_a4 o0 = {__builtin_bswap32(st[0]), __builtin_bswap32(st[1]), __builtin_bswap32(st[2]),
                 __builtin_bswap32(st[3])};
  u32x4_a4 o1 = {__builtin_bswap32(st[4]), __builtin_bswap32(st[5]), __builtin_bswap32(st[6]),
                 __builtin_bswap32(st[7])};
  *(u32x4_a4*)out = o0;
  *(u32x4_a4*)(out + 4) = o1;
}

// ---------------------------------------------------------------------------
// Interior node: SHA-256 of the 65 bytes 0x01 || L || R (two blocks).  L and R
// are digests as eight big-endian words, so the message words are L and R
// shifted right by one byte across word boundaries.
__device__ __forceinline__ void node_hash(const uint32_t (&L)[8], const uint32_t (&R)[8],
                                          uint32_t (&st)[8]) {
  sha256_init(st);
  uint32_t w[16];
  w[0] = 0x01000000u | (L[0] >> 8);
#pragma unroll
  for (int i = 1; i < 8; ++i) w[i] = __builtin_amdgcn_alignbit(L[i - 1], L[i], 8);
  w[8] = __builtin_amdgcn_alignbit(L[7], R[0], 8);
#pragma unroll
  for (int i = 9; i < 16; ++i) w[i] = __builtin_amdgcn_alignbit(R[i - 9], R[i - 8], 8);
  sha256_block(st, w);
  w[0] = (R[7] << 24) | 0x00800000u;
#pragma unroll
  for (int i = 1; i < 15; ++i) w[i] = 0;
  w[15] = 65 * 8;
  sha256_block(st, w);
}

__global__ __launch_bounds__(256) void hash_tree_kernel(const uint8_t* in, uint64_t n_in,
                                                        uint8_t* out) {
  __shared__ uint32_t s[2][kHashTreeFan][8];
  const uint32_t tid = threadIdx.x;
  if (n_in == 0) {  // no leaves: the hash of the empty message
    if (blockIdx.x == 0 && tid == 0) {
      uint32_t st[8], w[16];
      sha256_init(st);
      w[0] = 0x80000000u;
#pragma unroll
      for (int i = 1; i < 16; ++i) w[i] = 0;
      sha256_block(st, w);
#pragma unroll
      for (int i = 0; i < 8; ++i) ((uint32_t*)out)[i] = __builtin_bswap32(st[i]);
    }
    return;
  }
  const uint64_t base = (uint64_t)blockIdx.x * kHashTreeFan;
  uint32_t m = (uint32_t)(n_in - base < kHashTreeFan ? n_in - base : kHashTreeFan);
  const uint32_t* src = (const uint32_t*)(in + 32 * base);
  for (uint32_t i = tid; i < m * 8; i += blockDim.x)
    s[0][i >> 3][i & 7] = __builtin_bswap32(src[i]);
  __syncthreads();
  int cur = 0;
  // Pair neighbours level by level and carry an unpaired last node up as it
  // is: the same tree as RFC 6962's split at the largest power of two.
  while (m > 1) {
    const uint32_t half = (m + 1) / 2;
    if (tid < half) {
      uint32_t st[8];
      if (2 * tid + 1 < m) {
        uint32_t L[8], R[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          L[i] = s[cur][2 * tid][i];
          R[i] = s[cur][2 * tid + 1][i];
        }
        node_hash(L, R, st);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) st[i] = s[cur][2 * tid][i];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) s[cur ^ 1][tid][i] = st[i];
    }
    __syncthreads();
    cur ^= 1;
    m = half;
  }
  if (tid < 8) ((uint32_t*)(out + 32 * (uint64_t)blockIdx.x))[tid] = __builtin_bswap32(s[cur][0][tid]);
}

}  // namespace

hipError_t launch_hash_setup(const HashSetupParams& p, hipStream_t stream) {
  const uint32_t grid = p.njobs > 0 ? p.njobs : 1;
  hipLaunchKernelGGL(hash_setup_kernel, dim3(grid), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_hash_leaves(const HashLeafParams& p, hipStream_t stream) {
  if (p.nleaves == 0) return hipSuccess;
  const uint64_t grid = (p.nleaves + 255) / 256;
  hipLaunchKernelGGL(hash_leaf_kernel, dim3((uint32_t)grid), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_hash_tree(const uint8_t* in, uint64_t n_in, uint8_t* out, hipStream_t stream) {
  const uint64_t grid = n_in == 0 ? 1 : (n_in + kHashTreeFan - 1) / kHashTreeFan;
  hipLaunchKernelGGL(hash_tree_kernel, dim3((uint32_t)grid), dim3(256), 0, stream, in, n_in, out);
  return hipGetLastError();
}

}  // namespace pulse
