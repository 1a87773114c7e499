// gfx950 kernels of the replica state restore: pack + checksum, unpack +
// re-derive + verify, replica compare, checksum.
//
// All four are pure streaming (no reuse, integer arithmetic only), so the
// bound is HBM bandwidth.  Layout of the work:
//   * one unit = one chunk (or, for unpack, one bf16 parameter chunk together
//     with the two fp32 master chunks it is rounded from), processed by one
//     256-thread workgroup; units are taken in grid-stride order;
//   * each thread moves 16-byte vectors with non-temporal loads and stores,
//     kUnroll vectors in flight before the first is consumed;
//   * FRSUM-128 partial sums live in 64-bit registers per lane; a unit's
//     sums are folded across the wavefront with cross-lane shuffles and
//     across the four wavefronts through LDS (double-buffered, so one
//     barrier per unit);
//   * result sets are written with 32-bit atomic OR and a 64-bit atomic add,
//     whose outcome does not depend on the order of the units.
#include <hip/hip_runtime.h>

#include "fr_internal.h"

namespace fr {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned long long u64;

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr int kUnroll = 8;

__device__ __forceinline__ u32x4 ld_nt(const u32x4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_nt(u32x4 v, u32x4* p) { __builtin_nontemporal_store(v, p); }
__device__ __forceinline__ void st_nt2(u32x2 v, u32x2* p) { __builtin_nontemporal_store(v, p); }

// FRSUM-128 contribution of four consecutive words whose 0-based word index
// within the chunk starts at i0: sum += w, wsum += (index + 1) * w.
__device__ __forceinline__ void acc4(const u32x4& x, uint32_t i0, u64& s, u64& ws) {
  s += (u64)x.x + (u64)x.y + (u64)x.z + (u64)x.w;
  ws += (u64)(i0 + 1) * x.x + (u64)(i0 + 2) * x.y + (u64)(i0 + 3) * x.z + (u64)(i0 + 4) * x.w;
}

__device__ __forceinline__ void acc2(const u32x2& x, uint32_t i0, u64& s, u64& ws) {
  s += (u64)x.x + (u64)x.y;
  ws += (u64)(i0 + 1) * x.x + (u64)(i0 + 2) * x.y;
}

// fp32 bit pattern -> bf16 bit pattern, round to nearest, ties to even, in
// integer arithmetic (no flush of denormals): adding 0x7FFF plus the lowest
// kept bit carries into the kept half exactly when the dropped half is above
// the midpoint, or at it with an odd kept half.  NaN keeps its top bits with
// the quiet bit set.
__device__ __forceinline__ uint32_t rne_bf16(uint32_t u) {
  const uint32_t r = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
  return ((u & 0x7FFFFFFFu) > 0x7F800000u) ? ((u >> 16) | 0x40u) : r;
}

__device__ __forceinline__ u32x2 rne4(const u32x4& x) {
  return u32x2{rne_bf16(x.x) | (rne_bf16(x.y) << 16), rne_bf16(x.z) | (rne_bf16(x.w) << 16)};
}

// The first `t` bytes (t even, < 16) of a 16-byte-aligned vector, zero-filled;
// reads only those bytes.
__device__ __forceinline__ u32x4 load_tail(const uint8_t* p, uint32_t t) {
  const uint16_t* h = reinterpret_cast<const uint16_t*>(p);
  uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
  for (int b = 0; b < 7; b++)
    if (uint32_t(2 * b) < t) w[b >> 1] |= uint32_t(h[b]) << (16 * (b & 1));
  return u32x4{w[0], w[1], w[2], w[3]};
}

// Writes the first `t` bytes (t even, < 16) of x.
__device__ __forceinline__ void store_tail(uint8_t* p, const u32x4& x, uint32_t t) {
  uint16_t* h = reinterpret_cast<uint16_t*>(p);
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
  for (int b = 0; b < 7; b++)
    if (uint32_t(2 * b) < t) h[b] = uint16_t(w[b >> 1] >> (16 * (b & 1)));
}

// x with every byte at position >= t cleared (t even, < 16).
__device__ __forceinline__ u32x4 mask_tail(const u32x4& x, uint32_t t) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const uint32_t have = t > uint32_t(4 * i) ? t - 4 * i : 0;  // bytes of word i kept
    o[i] = have >= 4 ? w[i] : (have == 2 ? (w[i] & 0xFFFFu) : 0u);
  }
  return u32x4{o[0], o[1], o[2], o[3]};
}

// Sum K 64-bit values over the workgroup; every thread receives the totals.
// `lds` holds two buffers; alternating `parity` per unit makes one barrier
// enough (a buffer is rewritten only after the next unit's barrier, which all
// readers of the previous use have passed).
template <int K>
__device__ __forceinline__ void block_sum(u64 (&v)[K], u64 (&lds)[2][kWaves][K], int parity) {
#pragma unroll
  for (int k = 0; k < K; k++) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v[k] += __shfl_xor(v[k], o, 64);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < K; k++) lds[parity][wave][k] = v[k];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < K; k++) {
    u64 t = 0;
#pragma unroll
    for (int w = 0; w < kWaves; w++) t += lds[parity][w][k];
    v[k] = t;
  }
}

__device__ __forceinline__ void flag(uint32_t c, uint32_t* bitmap, u64* count) {
  atomicOr(bitmap + (c >> 5), 1u << (c & 31));
  atomicAdd(count, 1ull);
}

__device__ __forceinline__ bool differs(const fr_chunk_sum& want, u64 s, u64 ws) {
  return want.sum != s || want.wsum != ws;
}

// ------------------------------------------------------------------ pack

// kStore: pack (copy non-derived chunks into the payload); otherwise
// checksum only.  Every chunk's sums come from the bytes read at src.
template <bool kStore>
__global__ __launch_bounds__(kBlock) void k_pack(const ChunkRec* __restrict__ chunks,
                                                 uint32_t n_chunks,
                                                 const uint8_t* __restrict__ src,
                                                 uint8_t* __restrict__ payload,
                                                 fr_chunk_sum* __restrict__ sums) {
  __shared__ u64 lds[2][kWaves][2];
  int parity = 0;
  for (uint32_t c = blockIdx.x; c < n_chunks; c += gridDim.x, parity ^= 1) {
    const ChunkRec r = chunks[c];
    const u32x4* s = reinterpret_cast<const u32x4*>(src + r.src_off);
    const bool store = kStore && r.pay_off != kNoPayload;
    u32x4* d = reinterpret_cast<u32x4*>(payload + (store ? r.pay_off : 0));
    const uint32_t nvec = r.len >> 4;
    u64 acc[2] = {0, 0};
    uint32_t v = threadIdx.x;
    for (; v + (kUnroll - 1) * kBlock < nvec; v += kUnroll * kBlock) {
      u32x4 x[kUnroll];
#pragma unroll
      for (int q = 0; q < kUnroll; q++) x[q] = ld_nt(s + v + q * kBlock);
#pragma unroll
      for (int q = 0; q < kUnroll; q++) {
        acc4(x[q], 4 * (v + q * kBlock), acc[0], acc[1]);
        if (store) st_nt(x[q], d + v + q * kBlock);
      }
    }
    for (; v < nvec; v += kBlock) {
      const u32x4 x = ld_nt(s + v);
      acc4(x, 4 * v, acc[0], acc[1]);
      if (store) st_nt(x, d + v);
    }
    const uint32_t tail = r.len & 15;
    if (tail && threadIdx.x == nvec % kBlock) {
      const u32x4 x = load_tail(reinterpret_cast<const uint8_t*>(s + nvec), tail);
      acc4(x, 4 * nvec, acc[0], acc[1]);
      if (store) d[nvec] = x;  // the segment's zero padding is written with it
    }
    block_sum<2>(acc, lds, parity);
    if (threadIdx.x == 0) {
      sums[c].sum = acc[0];
      sums[c].wsum = acc[1];
    }
  }
}

// ---------------------------------------------------------------- unpack

__global__ __launch_bounds__(kBlock) void k_unpack(const ChunkRec* __restrict__ chunks,
                                                   const uint32_t* __restrict__ units,
                                                   uint32_t n_units, uint32_t cvec,
                                                   const uint8_t* __restrict__ payload,
                                                   const fr_chunk_sum* __restrict__ sums,
                                                   uint8_t* __restrict__ dst,
                                                   uint32_t* __restrict__ bitmap,
                                                   u64* __restrict__ n_bad) {
  __shared__ u64 lds[2][kWaves][6];
  int parity = 0;
  for (uint32_t u = blockIdx.x; u < n_units; u += gridDim.x, parity ^= 1) {
    const uint32_t c = units[u];
    const ChunkRec r = chunks[c];
    u64 acc[6] = {0, 0, 0, 0, 0, 0};
    if (r.master == kNoMaster) {
      // Plain chunk: copy, then check the bytes as written.
      const u32x4* s = reinterpret_cast<const u32x4*>(payload + r.pay_off);
      u32x4* d = reinterpret_cast<u32x4*>(dst + r.dst_off);
      const uint32_t nvec = r.len >> 4;
      uint32_t v = threadIdx.x;
      for (; v + (kUnroll - 1) * kBlock < nvec; v += kUnroll * kBlock) {
        u32x4 x[kUnroll];
#pragma unroll
        for (int q = 0; q < kUnroll; q++) x[q] = ld_nt(s + v + q * kBlock);
#pragma unroll
        for (int q = 0; q < kUnroll; q++) {
          st_nt(x[q], d + v + q * kBlock);
          acc4(x[q], 4 * (v + q * kBlock), acc[0], acc[1]);
        }
      }
      for (; v < nvec; v += kBlock) {
        const u32x4 x = ld_nt(s + v);
        st_nt(x, d + v);
        acc4(x, 4 * v, acc[0], acc[1]);
      }
      const uint32_t tail = r.len & 15;
      if (tail && threadIdx.x == nvec % kBlock) {
        // The payload segment is padded to 16 bytes, so the whole vector is
        // readable; only the entry's bytes are written and summed.
        const u32x4 x = mask_tail(s[nvec], tail);
        store_tail(reinterpret_cast<uint8_t*>(d + nvec), x, tail);
        acc4(x, 4 * nvec, acc[0], acc[1]);
      }
      block_sum<6>(acc, lds, parity);
      if (threadIdx.x == 0 && differs(sums[c], acc[0], acc[1])) flag(c, bitmap, n_bad);
    } else {
      // Derived group: bf16 parameter chunk c (r.len bytes) and the master
      // chunks m0 = r.master and m0 + 1 that hold its 2 * r.len source bytes.
      const uint32_t m0 = r.master;
      const ChunkRec m = chunks[m0];
      const uint32_t mbytes = 2 * r.len;
      const uint32_t nvm = mbytes >> 4;
      const u32x4* s = reinterpret_cast<const u32x4*>(payload + m.pay_off);
      u32x4* md = reinterpret_cast<u32x4*>(dst + m.dst_off);
      u32x2* pd = reinterpret_cast<u32x2*>(dst + r.dst_off);
      // Vectors [0, cvec) belong to master chunk m0, [cvec, nvm) to m0 + 1.
#pragma unroll
      for (int part = 0; part < 2; part++) {
        const uint32_t lo = part ? cvec : 0;
        const uint32_t hi = part ? nvm : (nvm < cvec ? nvm : cvec);
        u64& ms = acc[2 * part];
        u64& mws = acc[2 * part + 1];
        uint32_t v = lo + threadIdx.x;
        for (; v + (kUnroll - 1) * kBlock < hi; v += kUnroll * kBlock) {
          u32x4 x[kUnroll];
#pragma unroll
          for (int q = 0; q < kUnroll; q++) x[q] = ld_nt(s + v + q * kBlock);
#pragma unroll
          for (int q = 0; q < kUnroll; q++) {
            const uint32_t vv = v + q * kBlock;
            st_nt(x[q], md + vv);
            acc4(x[q], 4 * (vv - lo), ms, mws);
            const u32x2 p = rne4(x[q]);
            st_nt2(p, pd + vv);
            acc2(p, 2 * vv, acc[4], acc[5]);
          }
        }
        for (; v < hi; v += kBlock) {
          const u32x4 x = ld_nt(s + v);
          st_nt(x, md + v);
          acc4(x, 4 * (v - lo), ms, mws);
          const u32x2 p = rne4(x);
          st_nt2(p, pd + v);
          acc2(p, 2 * v, acc[4], acc[5]);
        }
      }
      const uint32_t tail = mbytes & 15;  // 0, 4, 8 or 12: whole fp32 values
      if (tail && threadIdx.x == nvm % kBlock) {
        const u32x4 x = mask_tail(s[nvm], tail);  // padded segment: readable
        uint8_t* mt = reinterpret_cast<uint8_t*>(md + nvm);
        uint32_t* mw = reinterpret_cast<uint32_t*>(mt);
        const uint32_t nf = tail >> 2;
        if (nf > 0) mw[0] = x.x;
        if (nf > 1) mw[1] = x.y;
        if (nf > 2) mw[2] = x.z;
        const int part = nvm < cvec ? 0 : 1;
        const uint32_t lo = part ? cvec : 0;
        acc4(x, 4 * (nvm - lo), acc[2 * part], acc[2 * part + 1]);
        uint16_t* ph = reinterpret_cast<uint16_t*>(pd + nvm);
        const uint32_t h0 = rne_bf16(x.x), h1 = rne_bf16(x.y), h2 = rne_bf16(x.z);
        if (nf > 0) ph[0] = uint16_t(h0);
        if (nf > 1) ph[1] = uint16_t(h1);
        if (nf > 2) ph[2] = uint16_t(h2);
        const u32x2 p{h0 | (nf > 1 ? h1 << 16 : 0u), nf > 2 ? h2 : 0u};
        acc2(p, 2 * nvm, acc[4], acc[5]);
      }
      block_sum<6>(acc, lds, parity);
      if (threadIdx.x == 0) {
        if (differs(sums[m0], acc[0], acc[1])) flag(m0, bitmap, n_bad);
        if (mbytes > 16 * cvec && differs(sums[m0 + 1], acc[2], acc[3])) flag(m0 + 1, bitmap, n_bad);
        if (differs(sums[c], acc[4], acc[5])) flag(c, bitmap, n_bad);
      }
    }
  }
}

// ---------------------------------------------------------------- verify

template <bool kSums>
__global__ __launch_bounds__(kBlock) void k_verify(const ChunkRec* __restrict__ chunks,
                                                   uint32_t n_chunks,
                                                   const uint8_t* __restrict__ a,
                                                   const uint8_t* __restrict__ b,
                                                   uint32_t* __restrict__ bitmap,
                                                   u64* __restrict__ n_diff,
                                                   fr_chunk_sum* __restrict__ sums_a,
                                                   fr_chunk_sum* __restrict__ sums_b) {
  __shared__ u64 lds[2][kWaves][4];
  constexpr int U = kSums ? kUnroll / 2 : kUnroll;
  int parity = 0;
  for (uint32_t c = blockIdx.x; c < n_chunks; c += gridDim.x, parity ^= 1) {
    const ChunkRec r = chunks[c];
    const u32x4* pa = reinterpret_cast<const u32x4*>(a + r.src_off);
    const u32x4* pb = reinterpret_cast<const u32x4*>(b + r.src_off);
    const uint32_t nvec = r.len >> 4;
    u64 acc[4] = {0, 0, 0, 0};
    uint32_t diff = 0;
    uint32_t v = threadIdx.x;
    for (; v + (U - 1) * kBlock < nvec; v += U * kBlock) {
      u32x4 xa[U], xb[U];
#pragma unroll
      for (int q = 0; q < U; q++) {
        xa[q] = ld_nt(pa + v + q * kBlock);
        xb[q] = ld_nt(pb + v + q * kBlock);
      }
#pragma unroll
      for (int q = 0; q < U; q++) {
        const u32x4 x = xa[q] ^ xb[q];
        diff |= x.x | x.y | x.z | x.w;
        if (kSums) {
          acc4(xa[q], 4 * (v + q * kBlock), acc[0], acc[1]);
          acc4(xb[q], 4 * (v + q * kBlock), acc[2], acc[3]);
        }
      }
    }
    for (; v < nvec; v += kBlock) {
      const u32x4 xa = ld_nt(pa + v), xb = ld_nt(pb + v);
      const u32x4 x = xa ^ xb;
      diff |= x.x | x.y | x.z | x.w;
      if (kSums) {
        acc4(xa, 4 * v, acc[0], acc[1]);
        acc4(xb, 4 * v, acc[2], acc[3]);
      }
    }
    const uint32_t tail = r.len & 15;
    if (tail && threadIdx.x == nvec % kBlock) {
      const u32x4 xa = load_tail(reinterpret_cast<const uint8_t*>(pa + nvec), tail);
      const u32x4 xb = load_tail(reinterpret_cast<const uint8_t*>(pb + nvec), tail);
      const u32x4 x = xa ^ xb;
      diff |= x.x | x.y | x.z | x.w;
      if (kSums) {
        acc4(xa, 4 * nvec, acc[0], acc[1]);
        acc4(xb, 4 * nvec, acc[2], acc[3]);
      }
    }
    // Any lane of any wave with a difference marks the chunk.
    const int hit = __syncthreads_or(int(diff != 0));
    if (kSums) block_sum<4>(acc, lds, parity);
    if (threadIdx.x == 0) {
      if (hit) flag(c, bitmap, n_diff);
      if (kSums) {
        sums_a[c].sum = acc[0];
        sums_a[c].wsum = acc[1];
        sums_b[c].sum = acc[2];
        sums_b[c].wsum = acc[3];
      }
    }
  }
}

// ------------------------------------------------------------- utilities

// Clears a result bitmap and its counter (a kernel rather than a memset so
// that the whole operation is made of kernel launches).
__global__ void k_zero(uint32_t* __restrict__ bitmap, uint64_t words, u64* __restrict__ count) {
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  for (uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < words; i += stride)
    bitmap[i] = 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) *count = 0;
}

inline uint32_t grid_for(uint64_t units, const LaunchCfg& cfg) {
  return uint32_t(units < cfg.max_grid ? units : cfg.max_grid);
}

inline int launch_zero(uint32_t* bitmap, uint64_t words, uint64_t* count, hipStream_t st) {
  const uint32_t blocks = uint32_t(words / 256 + 1 < 1024 ? words / 256 + 1 : 1024);
  hipLaunchKernelGGL(k_zero, dim3(blocks), dim3(256), 0, st, bitmap, words,
                     reinterpret_cast<u64*>(count));
  return int(hipGetLastError());
}

}  // namespace

int launch_pack(const ChunkRec* chunks, uint32_t n_chunks, const void* src, void* payload,
                fr_chunk_sum* sums, const LaunchCfg& cfg, void* stream) {
  if (n_chunks == 0) return 0;
  hipLaunchKernelGGL(k_pack<true>, dim3(grid_for(n_chunks, cfg)), dim3(kBlock), 0,
                     hipStream_t(stream), chunks, n_chunks,
                     static_cast<const uint8_t*>(src), static_cast<uint8_t*>(payload), sums);
  return int(hipGetLastError());
}

int launch_checksum(const ChunkRec* chunks, uint32_t n_chunks, const void* base,
                    fr_chunk_sum* sums, const LaunchCfg& cfg, void* stream) {
  if (n_chunks == 0) return 0;
  hipLaunchKernelGGL(k_pack<false>, dim3(grid_for(n_chunks, cfg)), dim3(kBlock), 0,
                     hipStream_t(stream), chunks, n_chunks,
                     static_cast<const uint8_t*>(base), static_cast<uint8_t*>(nullptr), sums);
  return int(hipGetLastError());
}

int launch_unpack(const ChunkRec* chunks, const uint32_t* units, uint32_t n_units, uint64_t C,
                  uint64_t bitmap_words, const void* payload, const fr_chunk_sum* sums,
                  void* dst, uint32_t* bitmap, uint64_t* n_bad, const LaunchCfg& cfg,
                  void* stream) {
  const hipStream_t st = hipStream_t(stream);
  int e = launch_zero(bitmap, bitmap_words, n_bad, st);
  if (e || n_units == 0) return e;
  hipLaunchKernelGGL(k_unpack, dim3(grid_for(n_units, cfg)), dim3(kBlock), 0, st, chunks, units,
                     n_units, uint32_t(C >> 4), static_cast<const uint8_t*>(payload), sums,
                     static_cast<uint8_t*>(dst), bitmap, reinterpret_cast<u64*>(n_bad));
  return int(hipGetLastError());
}

int launch_verify(const ChunkRec* chunks, uint32_t n_chunks, uint64_t bitmap_words,
                  const void* a, const void* b, uint32_t* bitmap, uint64_t* n_diff,
                  fr_chunk_sum* sums_a, fr_chunk_sum* sums_b, const LaunchCfg& cfg,
                  void* stream) {
  const hipStream_t st = hipStream_t(stream);
  int e = launch_zero(bitmap, bitmap_words, n_diff, st);
  if (e || n_chunks == 0) return e;
  const dim3 grid(grid_for(n_chunks, cfg));
  const auto* pa = static_cast<const uint8_t*>(a);
  const auto* pb = static_cast<const uint8_t*>(b);
  u64* nd = reinterpret_cast<u64*>(n_diff);
  if (sums_a)
    hipLaunchKernelGGL(k_verify<true>, grid, dim3(kBlock), 0, st, chunks, n_chunks, pa, pb,
                       bitmap, nd, sums_a, sums_b);
  else
    hipLaunchKernelGGL(k_verify<false>, grid, dim3(kBlock), 0, st, chunks, n_chunks, pa, pb,
                       bitmap, nd, sums_a, sums_b);
  return int(hipGetLastError());
}

}  // namespace fr
