// gfx950 kernels of the replica state restore: pack + checksum, unpack +
// re-derive + verify, replica compare, checksum.
//
// All four are pure streaming (no reuse, integer arithmetic only), so the
// bound is HBM bandwidth, and what decides the achieved bandwidth is how the
// waves' accesses are spread over memory.  Measured on MI355X: a copy in
// which each workgroup streams its own 64 KiB region (thousands of
// concurrent sequential streams) saturates near 5.3-5.5 TB/s, while the same
// copy cut into 4-8 KiB slices, one slice per workgroup and workgroups
// launched in address order, keeps the whole chip working inside one compact
// window and reaches 6.5-6.7 TB/s.  So:
//   * the unit of work is a slice of SL = min(tile, C) bytes of one chunk
//     (tile = B threads x U vectors x 16 B); a slot table lists the slices
//     of every unit in address order, one per workgroup id, so launch order
//     is table (address) order and no workgroup is idle (a workgroup reads
//     its slot, then its unit's record, then its data);
//   * each thread moves U 16-byte vectors with non-temporal loads/stores;
//   * FRSUM-128 is additive over any split of a chunk when every word keeps
//     its absolute index, so a slice sums its words with their chunk-relative
//     indices, folds the totals over the workgroup (cross-lane shuffles, then
//     LDS), and one thread adds them into 64-bit accumulators with atomics
//     (order-independent, hence deterministic);
//   * atomics on one address serialise, so no accumulator takes more than
//     16 slices (32 for a bf16 parameter fed by master slices): a chunk of
//     SPC slices owns G = max(1, SPC / 16) accumulators in the plan's
//     scratch, cleared by a fill kernel launched first;
//   * replica compare marks a differing chunk with a plain store of 1 to a
//     per-chunk flag (idempotent, so no atomics on shared bitmap words);
//   * for tensors that start inside a cache line, pack and unpack walk
//     tiles of the side they write instead of slices of chunks: workgroup g
//     writes one aligned tile of the payload (pack) or of the receiver arena
//     (unpack), across chunk and entry boundaries, summing each chunk's part
//     with the chunk's own word indices (k_pack_blocks, k_unpack_blocks);
//     the compare cuts its slices at lines of the arenas so that no line is
//     read by two workgroups (the checksum measured slower that way); other
//     line-aligned slice walks remain options (the plan's launch
//     configuration sets all of it per operation, see LaunchCfg);
//   * a finalize kernel, one lane per chunk, folds the G accumulators into
//     the chunk's sums (pack, checksum, compare) or compares them with the
//     sums sent (unpack; and, given two replicas' sums as accumulators and
//     as the sums sent, the consistency check from sums alone), and writes
//     whole bitmap words from wave ballots.
// Plan creation uses one more kernel: the host describes each slot table as
// one run of slots per unit and k_expand_slots writes the table itself.
// Delta calls build their lists' unit records on the device (k_list_*,
// below), so that a repair can follow the compare with no host work.
#include <hip/hip_runtime.h>

#include <mutex>

#include "fr_internal.h"

namespace fr {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned long long u64;

__device__ __forceinline__ u32x4 ld_nt(const u32x4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_nt(u32x4 v, u32x4* p) { __builtin_nontemporal_store(v, p); }
__device__ __forceinline__ void st_nt2(u32x2 v, u32x2* p) { __builtin_nontemporal_store(v, p); }

// Raw buffer accesses: a resource describes `bytes` bytes from `base`
// (stride 0, the gfx9 family's default format word); a 16-byte load at a
// byte offset at or past `bytes` returns zeros and a store there is dropped,
// with no memory access.  Every lane then issues its loads unconditionally,
// so nothing waits on a load before all of a thread's loads are in flight.
// Cache policy 2 is the non-temporal hint.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOob = 0xFFFFFFF0u;  // an offset past every range used here
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), short(0), int(bytes), 0x00020000);
}
__device__ __forceinline__ u32x4 ld_buf(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, int(off), 0, 2);
}
__device__ __forceinline__ void st_buf(const u32x4& v, rsrc_t r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, int(off), 0, 2);
}

// Thread's vectors q (slice vector l = q B + threadIdx.x, unit vector
// v0 + l) of a slice of sl_vec vectors of a unit whose nvec whole vectors
// start at s.  Vectors outside [0, nvec) (a lead wraps v0 + l past it) or
// past the slice are zeros (kBuf) or left unset (callers use only the
// others).
template <int B, int U, bool kBuf>
__device__ __forceinline__ void load_slice(u32x4 (&x)[U], const u32x4* s, uint32_t nvec, uint32_t v0,
                                           uint32_t sl_vec) {
  if constexpr (kBuf) {
    const rsrc_t in = make_rsrc(s, 16 * nvec);
#pragma unroll
    for (int q = 0; q < U; q++) {
      const uint32_t l = q * B + threadIdx.x;
      x[q] = ld_buf(in, l < sl_vec ? 16 * (v0 + l) : kOob);
    }
  } else {
#pragma unroll
    for (int q = 0; q < U; q++) {
      const uint32_t l = q * B + threadIdx.x, v = v0 + l;
      if (l < sl_vec && v < nvec) x[q] = ld_nt(s + v);
    }
  }
}

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

// v plus the v of lane (i op CTRL) for a DPP lane pattern that reads a
// lane for every lane: the halves moved across lanes (no old value kept),
// then added as 32-bit halves with a carry (fewer instructions than a
// 64-bit move and add).
template <int CTRL>
__device__ __forceinline__ u64 add_dpp(u64 v) {
  const uint32_t lo = uint32_t(v), hi = uint32_t(v >> 32);
  const uint32_t plo = uint32_t(__builtin_amdgcn_mov_dpp(int(lo), CTRL, 0xF, 0xF, false));
  const uint32_t phi = uint32_t(__builtin_amdgcn_mov_dpp(int(hi), CTRL, 0xF, 0xF, false));
  const uint32_t rlo = lo + plo;
  const uint32_t rhi = hi + phi + (rlo < lo ? 1u : 0u);
  return (u64(rhi) << 32) | rlo;
}

__device__ __forceinline__ u64 readlane64(u64 v, int lane) {
  const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v)), lane));
  const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v >> 32)), lane));
  return (u64(hi) << 32) | lo;
}

// Sum of a 64-bit value over the 64 lanes of a wave (uniform result).
// Within each row of 16 lanes: swap neighbours, swap pairs (quad_perm
// [1,0,3,2] and [2,3,0,1]) then rotate the row by 4 and by 8, after which
// every lane of a row holds the row's total; the four row totals are then
// read into scalar registers and added.
__device__ __forceinline__ u64 wave_sum(u64 v) {
  v = add_dpp<0xB1>(v);   // quad_perm [1,0,3,2]
  v = add_dpp<0x4E>(v);   // quad_perm [2,3,0,1]
  v = add_dpp<0x124>(v);  // row_ror:4
  v = add_dpp<0x128>(v);  // row_ror:8
  return readlane64(v, 0) + readlane64(v, 16) + readlane64(v, 32) + readlane64(v, 48);
}

// Sum K 64-bit values over the workgroup; thread 0 receives the totals.
// Several waves combine through LDS; `lds` holds two buffers, and callers
// flip `parity` after every call, so that one barrier per call is enough
// when a workgroup walks several slices: a wave writes buffer p again only
// after the barrier of the call in between, which thread 0 passes only once
// it has read buffer p.  (Flipping per loop iteration instead would break
// this when an iteration skips its call: two calls in a row would then use
// the same buffer with no barrier between thread 0's reads and the next
// writes.)
template <int B, int K>
__device__ __forceinline__ void block_sum(u64 (&v)[K], u64 (&lds)[2][B / 64][K], int parity) {
#pragma unroll
  for (int k = 0; k < K; k++) v[k] = wave_sum(v[k]);
  if (B == 64) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < K; k++) lds[parity][wave][k] = v[k];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
#pragma unroll
    for (int k = 0; k < K; k++) {
      u64 t = 0;
#pragma unroll
      for (int w = 0; w < B / 64; w++) t += lds[parity][w][k];
      v[k] = t;
    }
  }
}

__device__ __forceinline__ void add_sum(fr_chunk_sum* acc, u64 s, u64 ws) {
  atomicAdd(reinterpret_cast<u64*>(&acc->sum), s);
  atomicAdd(reinterpret_cast<u64*>(&acc->wsum), ws);
}

// Geometry of the slice walk shared by the kernels.
struct Walk {
  const u64* slots;   // slot table, XCD-major (see SlotTable); NULL: implicit
  u64 n_slices;       // workgroup ids to cover: slots in the walk
  u64 stride;         // entries per XCD in the table
  uint32_t imp_shift; // implicit walk: log2 of the slots per unit
  uint32_t sl_vec;    // vectors per slice: SL / 16
  uint32_t spc_shift; // log2(SPC), slices per chunk
  uint32_t g_shift;   // log2(G), accumulators per chunk
  uint32_t line;      // line-aligned walk: 1 at arena lines, 2 at payload lines (SlotTable::shift)
  uint32_t absorb;    // line-aligned walk: the last slice of a unit takes its leftover lead
  const u64* count;   // implicit walk of a list built on the device: its number of units
};

// Workgroup ids a launch covers: every slot of the walk, or for a list
// built on the device (whose length the host does not know) the slots of
// its first *count units.
__device__ __forceinline__ u64 walk_slices(const Walk& wk) {
  if (!wk.count) return wk.n_slices;
  const u64 n = *wk.count << wk.imp_shift;
  return n < wk.n_slices ? n : wk.n_slices;
}

// Vectors a line-aligned walk starts a unit's slices early (0 for a plain
// walk): the unit's offset into a line of the arena (mode 1) or of the
// payload (2), or into a slice of the payload (3).
__device__ __forceinline__ uint32_t lead_vectors(const Walk& wk, uint32_t lead, uint32_t plead) {
  const uint32_t b = wk.line == 1   ? lead % kLine
                     : wk.line == 2 ? plead % kLine
                     : wk.line == 3 ? plead & ((wk.sl_vec << 4) - 1)
                                    : 0u;
  return b >> 4;
}

// Slot of workgroup id g: (unit << 32) | j.
__device__ __forceinline__ u64 slot_of(const Walk& wk, u64 g) {
  if (wk.slots) return wk.slots[(g & 7) * wk.stride + (g >> 3)];
  return ((g >> wk.imp_shift) << 32) | (g & ((u64(1) << wk.imp_shift) - 1));
}

constexpr uint32_t kAccSlicesShift = 4;  // 16 slices per accumulator

// Accumulator of slice j of chunk c.  A line-aligned walk can give a chunk
// one slice more than SPC; that slice shares the chunk's last accumulator.
__device__ __forceinline__ u64 acc_index(const Walk& wk, uint32_t c, uint32_t j) {
  const uint32_t a = j >> kAccSlicesShift, last = (1u << wk.g_shift) - 1;
  return (u64(c) << wk.g_shift) + (a < last ? a : last);
}

// ------------------------------------------------------------------ pack

// kStore: pack (copy non-derived chunks into the payload); otherwise
// checksum only.  Sums of the bytes read at src go to acc (zeroed), every
// chunk's own accumulators; derived entries are read and summed only.
// kBuf: the slices' loads through a buffer resource (all in flight at
// once), else predicated global loads.
template <int B, int U, bool kStore, bool kBuf>
__global__ __launch_bounds__(B) void k_pack(const SrcUnit* __restrict__ units, Walk wk,
                                            const uint8_t* __restrict__ src,
                                            uint8_t* __restrict__ payload,
                                            fr_chunk_sum* __restrict__ acc_out) {
  __shared__ u64 lds[2][B / 64][2];
  int parity = 0;
  const u64 n_slices = walk_slices(wk);
  for (u64 g = blockIdx.x; g < n_slices; g += gridDim.x) {
    const u64 e = slot_of(wk, g);
    const SrcUnit r = units[e >> 32];
    const uint32_t c = r.c, j = uint32_t(e);
    const uint32_t nvec = r.len >> 4, tail = r.len & 15;
    const uint32_t endv = nvec + (tail ? 1u : 0u);
    // First vector of the slice; a line-aligned walk starts it lead_v
    // vectors early (the first slice's leading lanes then come before the
    // chunk: their unsigned index wraps past nvec and they do nothing).
    const uint32_t lead_v = lead_vectors(wk, r.lead, r.plead);
    const uint32_t v0 = j * wk.sl_vec - lead_v;
    if (j * wk.sl_vec >= endv + lead_v) continue;  // guard: no listed slot is empty
    // Vectors of the slice: a whole slice, except that a walk that absorbs
    // the lead gives the chunk's last slice everything up to its end (up to
    // lead_v vectors more than a slice) instead of one more, nearly empty,
    // slice.
    const bool last = (j + 1) * wk.sl_vec >= endv + (wk.absorb ? 0u : lead_v);
    const uint32_t n = last && wk.absorb ? endv - v0 : wk.sl_vec;
    const u32x4* s = reinterpret_cast<const u32x4*>(src + r.src_off);
    const bool store = kStore && r.pay_off != kNoPayload;
    u32x4* d = reinterpret_cast<u32x4*>(payload + (store ? r.pay_off : 0));
    u64 acc[2] = {0, 0};
    u32x4 x[U];
    load_slice<B, U, kBuf>(x, s, nvec, v0, wk.sl_vec);
  #pragma unroll
    for (int q = 0; q < U; q++) {
      const uint32_t l = q * B + threadIdx.x, v = v0 + l;
      if (l < wk.sl_vec && v < nvec) {
        acc4(x[q], 4 * v, acc[0], acc[1]);
        if (store) st_nt(x[q], d + v);
      }
    }
    for (uint32_t l = wk.sl_vec + threadIdx.x; l < n; l += B) {  // an absorbing last slice
      const uint32_t v = v0 + l;
      if (v < nvec) {
        const u32x4 y = ld_nt(s + v);
        acc4(y, 4 * v, acc[0], acc[1]);
        if (store) st_nt(y, d + v);
      }
    }
    if (tail && nvec - v0 < n && threadIdx.x == (nvec - v0) % B) {
      const u32x4 t = load_tail(reinterpret_cast<const uint8_t*>(s + nvec), tail);
      acc4(t, 4 * nvec, acc[0], acc[1]);
      if (store) d[nvec] = t;  // the segment's zero padding is written with it
    }
    // The chunk's last slice zero-fills the gap up to the next payload
    // segment (fewer than segment alignment / 16 vectors).
    if (store && r.gap_v && last) {
      for (uint32_t v = endv + threadIdx.x; v < endv + r.gap_v; v += B)
        st_nt(u32x4{0, 0, 0, 0}, d + v);
    }
    block_sum<B, 2>(acc, lds, parity);
    parity ^= 1;
    if (threadIdx.x == 0) add_sum(acc_out + acc_index(wk, c, j), acc[0], acc[1]);
  }
}

// Pack walked by blocks of the payload: workgroup b writes the payload's
// vectors [b T, (b + 1) T) (T = B U, the tile), whatever chunks they belong
// to, so that every workgroup stores one whole aligned tile of the payload
// even where segments start inside lines.  Vector o of the payload belongs to
// the last sent chunk u with u.pay_off / 16 <= o: its data, its ragged tail
// (zero-padded) or the zero gap after it.  A block's chunks are found from
// the first one (`first`, XCD-major like a slot table) on; its sums are
// reduced once per chunk it touches.  The chunks without payload (derived
// entries: read and summed only) are walked by k_pack in a launch of their
// own.
struct PackBlocksArgs {
  const SrcUnit* pay_units;  // sent chunks in payload order
  const uint32_t* first;     // per block, XCD-major: index of the unit holding its first vector
  u64 n_units, n_blocks, stride, pay_vecs;
};

template <int B, int U>
__device__ __forceinline__ void pack_block(const PackBlocksArgs& a, const Walk& wk, u64 b,
                                           const uint8_t* __restrict__ src,
                                           uint8_t* __restrict__ payload,
                                           fr_chunk_sum* __restrict__ acc_out,
                                           u64 (&lds)[2][B / 64][2], int& parity) {
  constexpr uint32_t T = B * U;
  const u64 v_blk = b * T;
  // vectors of this block (T except in the last one); a thread's vector q is
  // the block's vector l = q B + threadIdx.x, payload vector v_blk + l
  const uint32_t n_here = uint32_t(v_blk + T < a.pay_vecs ? T : a.pay_vecs - v_blk);
  const u64 v_end = v_blk + n_here;
  const rsrc_t out = make_rsrc(payload + 16 * v_blk, 16 * n_here);
  const u64 u0 = a.first[(b & 7) * a.stride + (b >> 3)];
  // The block's units from u0 on, one pass each: block vectors [lb, le) of
  // unit u are its vectors from du on.  Its data vectors are read through a
  // resource that ends before its ragged tail (so the tail and the gap after
  // the unit load as zeros), and the tail's thread reads the tail's bytes.
  // (Loading two units' vectors together measured slower on the descriptor
  // stress table: 5.70 against 5.77 TB/s.)
  u64 u = u0;
  uint32_t lb = 0;
  while (true) {
    const SrcUnit r = a.pay_units[u];
    const u64 pn = u + 1 < a.n_units ? (a.pay_units[u + 1].pay_off >> 4) : a.pay_vecs;
    const uint32_t le = pn < v_end ? uint32_t(pn - v_blk) : n_here;
    const uint32_t du = u == u0 ? uint32_t(v_blk - (r.pay_off >> 4)) : 0u;
    const uint32_t nvec = r.len >> 4;
    const rsrc_t in = make_rsrc(src + r.src_off, 16 * nvec);
    u32x4 x[U];
#pragma unroll
    for (int q = 0; q < U; q++) {
      const uint32_t l = q * B + threadIdx.x;
      x[q] = ld_buf(in, l >= lb && l < le ? 16 * (l - lb + du) : kOob);
    }
    const uint32_t lt = nvec - du + lb;  // block vector of the ragged tail
    const bool tail = (r.len & 15) && nvec >= du && lt < le;
    u32x4 tv = u32x4{0, 0, 0, 0};
    if (tail && threadIdx.x == lt % B) tv = load_tail(src + r.src_off + 16 * u64(nvec), r.len & 15);
    u64 t[2] = {0, 0};
#pragma unroll
    for (int q = 0; q < U; q++) {
      const uint32_t l = q * B + threadIdx.x;
      if (tail && l == lt) x[q] = tv;
      if (l >= lb && l < le) {
        st_buf(x[q], out, 16 * l);
        acc4(x[q], 4 * (l - lb + du), t[0], t[1]);  // zeros (gap) add nothing
      }
    }
    block_sum<B, 2>(t, lds, parity);
    parity ^= 1;
    if (threadIdx.x == 0) add_sum(acc_out + acc_index(wk, r.c, du / wk.sl_vec), t[0], t[1]);
    if (le >= n_here) break;
    u++;
    lb = le;
  }
}

template <int B, int U>
__global__ __launch_bounds__(B) void k_pack_blocks(PackBlocksArgs a, Walk wk,
                                                   const uint8_t* __restrict__ src,
                                                   uint8_t* __restrict__ payload,
                                                   fr_chunk_sum* __restrict__ acc_out) {
  __shared__ u64 lds[2][B / 64][2];
  int parity = 0;
  for (u64 g = blockIdx.x; g < a.n_blocks; g += gridDim.x)
    pack_block<B, U>(a, wk, g, src, payload, acc_out, lds, parity);
}

// First unit of every payload block (see k_pack_blocks): the last unit
// starting at or before the block's first vector, by binary search over the
// units' payload offsets (pay_off[4 u]: 32-byte unit records); written
// XCD-major, zero past the blocks.
__global__ __launch_bounds__(256) void k_block_first(const u64* __restrict__ pay_off, u64 n_units,
                                                     u64 n_blocks, u64 stride, uint32_t block_vecs,
                                                     uint32_t* __restrict__ out) {
  const u64 total = 8 * stride;
  for (u64 b = u64(blockIdx.x) * blockDim.x + threadIdx.x; b < total;
       b += u64(gridDim.x) * blockDim.x) {
    uint32_t v = 0;
    if (b < n_blocks) {
      const u64 o = b * block_vecs;
      u64 lo = 0, hi = n_units;  // the first unit starts the payload: pay_off 0 <= o
      while (hi - lo > 1) {
        const u64 mid = (lo + hi) / 2;
        if ((pay_off[4 * mid] >> 4) <= o) lo = mid;
        else hi = mid;
      }
      v = uint32_t(lo);
    }
    out[(b & 7) * stride + (b >> 3)] = v;
  }
}

// ---------------------------------------------------------------- unpack

// Two kinds of units, listed by the walk in payload order (a derived group
// where its entry stands in the table):
//   derived: bf16 parameter chunk c and the master chunks m0 = master(c) and
//            m0 + 1 holding its 2 * len source bytes; walked in slices of
//            master bytes (at most 2 * SPC per unit), each slice inside one
//            master chunk;
//   plain:   a chunk of an entry that is neither derived nor a master with a
//            derived image; at most SPC slices per unit.
// Sums of the bytes written go to the accumulators `acc_out` (zeroed).
// One slice of a derived group: read master bytes from `msrc` (the payload,
// or with kFromPayload = false the receiver's own masters), write the bf16
// images to the parameter chunk, and with kFromPayload also write the master
// bytes to the receiver.  acc[0..1] get the master words' sums (relative to
// master chunk m0 + part), acc[2..3] the parameter words'.  Returns false
// for a slice past the group's end.
template <int B, int U, bool kFromPayload, bool kBuf>
__device__ __forceinline__ bool derived_slice(const DerivedUnit& r, uint32_t j, const Walk& wk,
                                              uint32_t cvec, const uint8_t* msrc, uint8_t* dst,
                                              u64 (&acc)[4], uint32_t& part) {
  const uint32_t mvec = (2 * r.len) >> 4;  // whole master vectors of the group
  const uint32_t mtail = (2 * r.len) & 15;  // 0, 4, 8 or 12: whole fp32 values
  const uint32_t v0 = j * wk.sl_vec;
  if (v0 > mvec || (v0 == mvec && mtail == 0)) return false;
  part = j >> wk.spc_shift;                 // master chunk of this slice: m0 + part
  const uint32_t wbase = part * cvec * 4;   // its first word in the group
  const u32x4* s = reinterpret_cast<const u32x4*>(msrc + r.m_pay_off);
  u32x4* md = reinterpret_cast<u32x4*>(dst + r.m_dst_off);
  u32x2* pd = reinterpret_cast<u32x2*>(dst + r.p_dst_off);
  u32x4 x[U];
  load_slice<B, U, kBuf>(x, s, mvec, v0, wk.sl_vec);
#pragma unroll
  for (int q = 0; q < U; q++) {
    const uint32_t l = q * B + threadIdx.x, v = v0 + l;
    if (l < wk.sl_vec && v < mvec) {
      if (kFromPayload) {
        st_nt(x[q], md + v);
        acc4(x[q], 4 * v - wbase, acc[0], acc[1]);
      }
      const u32x2 p = rne4(x[q]);
      st_nt2(p, pd + v);
      acc2(p, 2 * v, acc[2], acc[3]);
    }
  }
  if (mtail && mvec >= v0 && mvec - v0 < wk.sl_vec && threadIdx.x == (mvec - v0) % B) {
    // A payload segment is padded to 16 bytes, so its whole last vector is
    // readable; the receiver's master is read only up to its last value.
    const u32x4 t = kFromPayload ? mask_tail(s[mvec], mtail)
                                 : load_tail(reinterpret_cast<const uint8_t*>(s + mvec), mtail);
    const uint32_t nf = mtail >> 2;
    if (kFromPayload) {
      uint32_t* mw = reinterpret_cast<uint32_t*>(md + mvec);
      mw[0] = t.x;
      if (nf > 1) mw[1] = t.y;
      if (nf > 2) mw[2] = t.z;
      acc4(t, 4 * mvec - wbase, acc[0], acc[1]);
    }
    uint16_t* ph = reinterpret_cast<uint16_t*>(pd + mvec);
    const uint32_t h0 = rne_bf16(t.x), h1 = rne_bf16(t.y), h2 = rne_bf16(t.z);
    ph[0] = uint16_t(h0);
    if (nf > 1) ph[1] = uint16_t(h1);
    if (nf > 2) ph[2] = uint16_t(h2);
    const u32x2 p{h0 | (nf > 1 ? h1 << 16 : 0u), nf > 2 ? h2 : 0u};
    acc2(p, 2 * mvec, acc[2], acc[3]);
  }
  return true;
}

// One slice of a plain chunk: copy, and sum the bytes as written.  A walk
// cut at slice boundaries of the payload (mode 3) starts the chunk's slices
// lead_v vectors early (the first slice's leading lanes then come before the
// chunk: their unsigned index wraps past nvec and they do nothing).
template <int B, int U, bool kBuf>
__device__ __forceinline__ bool plain_slice(const PlainUnit& r, uint32_t j, const Walk& wk,
                                            const uint8_t* payload, uint8_t* dst,
                                            u64 (&acc)[2]) {
  const uint32_t nvec = r.len >> 4, tail = r.len & 15, endv = nvec + (tail ? 1u : 0u);
  const uint32_t lead_v = lead_vectors(wk, r.dlead, r.plead);
  if (j * wk.sl_vec >= endv + lead_v) return false;
  const uint32_t v0 = j * wk.sl_vec - lead_v;
  // as in k_pack: an absorbing walk's last slice runs to the chunk's end
  const bool last = (j + 1) * wk.sl_vec >= endv + (wk.absorb ? 0u : lead_v);
  const uint32_t n = last && wk.absorb ? endv - v0 : wk.sl_vec;
  const u32x4* s = reinterpret_cast<const u32x4*>(payload + r.pay_off);
  u32x4* d = reinterpret_cast<u32x4*>(dst + r.dst_off);
  u32x4 x[U];
  load_slice<B, U, kBuf>(x, s, nvec, v0, wk.sl_vec);
#pragma unroll
  for (int q = 0; q < U; q++) {
    const uint32_t l = q * B + threadIdx.x, v = v0 + l;
    if (l < wk.sl_vec && v < nvec) {
      st_nt(x[q], d + v);
      acc4(x[q], 4 * v, acc[0], acc[1]);
    }
  }
  for (uint32_t l = wk.sl_vec + threadIdx.x; l < n; l += B) {  // an absorbing last slice
    const uint32_t v = v0 + l;
    if (v < nvec) {
      const u32x4 y = ld_nt(s + v);
      st_nt(y, d + v);
      acc4(y, 4 * v, acc[0], acc[1]);
    }
  }
  if (tail && nvec - v0 < n && threadIdx.x == (nvec - v0) % B) {
    // The payload segment is padded to 16 bytes, so the whole vector is
    // readable; only the entry's bytes are written and summed.
    const u32x4 t = mask_tail(s[nvec], tail);
    store_tail(reinterpret_cast<uint8_t*>(d + nvec), t, tail);
    acc4(t, 4 * nvec, acc[0], acc[1]);
  }
  return true;
}

template <int B, int U, bool kBuf>
__global__ __launch_bounds__(B) void k_unpack(const DerivedUnit* __restrict__ derived,
                                              const PlainUnit* __restrict__ plain, Walk wk,
                                              uint32_t cvec, const uint8_t* __restrict__ payload,
                                              uint8_t* __restrict__ dst,
                                              fr_chunk_sum* __restrict__ acc_out) {
  __shared__ u64 lds[2][B / 64][4];
  __shared__ u64 lds2[2][B / 64][2];
  int parity = 0;
  const u64 n_slices = walk_slices(wk);
  for (u64 g = blockIdx.x; g < n_slices; g += gridDim.x) {
    const u64 e = slot_of(wk, g);
    if (uint32_t(e) & kSlotDerived) {
      const DerivedUnit r = derived[e >> 32];
      const uint32_t j = uint32_t(e) & ~kSlotDerived;
      u64 acc[4] = {0, 0, 0, 0};
      uint32_t part = 0;
      if (!derived_slice<B, U, true, kBuf>(r, j, wk, cvec, payload, dst, acc, part)) continue;
      block_sum<B, 4>(acc, lds, parity);
      parity ^= 1;
      if (threadIdx.x == 0) {
        const uint32_t jj = j - (part << wk.spc_shift);  // slice within its master chunk
        add_sum(acc_out + ((u64(r.m0 + part) << wk.g_shift) + (jj >> kAccSlicesShift)), acc[0],
                acc[1]);
        // a parameter accumulator covers 16 slices' worth of parameter bytes,
        // which come from 32 master slices
        add_sum(acc_out + ((u64(r.c) << wk.g_shift) + (j >> (kAccSlicesShift + 1))), acc[2],
                acc[3]);
      }
    } else {
      const PlainUnit r = plain[e >> 32];
      const uint32_t j = uint32_t(e);
      u64 acc[2] = {0, 0};
      if (!plain_slice<B, U, kBuf>(r, j, wk, payload, dst, acc)) continue;
      block_sum<B, 2>(acc, lds2, parity);
      parity ^= 1;
      if (threadIdx.x == 0) add_sum(acc_out + acc_index(wk, r.c, j), acc[0], acc[1]);
    }
  }
}

// Unpack walked by blocks of the receiver (for tables whose receiver chunks
// start inside lines): workgroup g writes the plain chunks' bytes inside one
// aligned tile of the receiver arena (T = B U vectors), so that no line is
// written by two workgroups and every workgroup's writes fall in one
// aligned tile; the gaps between entries are not touched.  Only tiles that
// hold some chunk bytes are listed.  A chunk's data is read from its payload
// segment and summed with its chunk-relative word indices; its ragged tail
// is masked to its bytes (the payload's padding is not trusted).  The
// derived groups (which write their masters too) are walked by k_unpack in
// a launch of their own.
struct UnpackBlocksArgs {
  const PlainUnit* units;  // plain chunks in receiver order
  const u64* blocks;       // listed tiles, XCD-major: (tile index << 32) | first unit touching it
  u64 n_units, n_blocks, stride;
};

// One unit's part of a receiver tile: the unit's vectors from du on are the
// tile's vectors from lb on.  Its ragged tail (if in the tile) is masked to
// its bytes, written and added to t by the thread holding it.
__device__ __forceinline__ void unpack_tile_tail(const PlainUnit& r, uint32_t lb, uint32_t du,
                                                 uint32_t T, uint32_t B, const uint8_t* payload,
                                                 uint8_t* dst, u64 (&t)[2]) {
  const uint32_t nvec = r.len >> 4, tail = r.len & 15;
  const uint32_t lt = nvec - du + lb;  // tile vector of the ragged tail
  if (tail && nvec >= du && lt < T && threadIdx.x == lt % B) {
    const u32x4 tv = mask_tail(ld_nt(reinterpret_cast<const u32x4*>(payload + r.pay_off) + nvec), tail);
    store_tail(dst + r.dst_off + 16 * u64(nvec), tv, tail);
    acc4(tv, 4 * nvec, t[0], t[1]);
  }
}

template <int B, int U>
__global__ __launch_bounds__(B) void k_unpack_blocks(UnpackBlocksArgs a, Walk wk,
                                                     const uint8_t* __restrict__ payload,
                                                     uint8_t* __restrict__ dst,
                                                     fr_chunk_sum* __restrict__ acc_out) {
  constexpr uint32_t T = B * U;
  __shared__ u64 lds[2][B / 64][2];
  int parity = 0;
  for (u64 g = blockIdx.x; g < a.n_blocks; g += gridDim.x) {
    const u64 e = a.blocks[(g & 7) * a.stride + (g >> 3)];
    const u64 v_blk = (e >> 32) * T, v_end = v_blk + T;  // receiver vectors of the tile
    const u64 u0 = uint32_t(e);
    const PlainUnit r0 = a.units[u0];
    const u64 dv0 = r0.dst_off >> 4;
    const uint32_t lb0 = dv0 > v_blk ? uint32_t(dv0 - v_blk) : 0u;
    const uint32_t du0 = v_blk > dv0 ? uint32_t(v_blk - dv0) : 0u;
    const bool two = u0 + 1 < a.n_units && (a.units[u0 + 1].dst_off >> 4) < v_end;
    const bool many = two && u0 + 2 < a.n_units && (a.units[u0 + 2].dst_off >> 4) < v_end;
    if (!many) {
      // One or two units, the common case: both units' loads in flight
      // together.  A thread's vector belongs to unit 1 from lb1 on; every
      // other vector outside a unit's data loads as zero and is not stored.
      const PlainUnit r1 = two ? a.units[u0 + 1] : r0;
      const uint32_t lb1 = two ? uint32_t((r1.dst_off >> 4) - v_blk) : T;
      const rsrc_t in0 = make_rsrc(payload + r0.pay_off, 16 * (r0.len >> 4));
      const rsrc_t out0 = make_rsrc(dst + r0.dst_off, 16 * (r0.len >> 4));
      u32x4 x[U];
#pragma unroll
      for (int q = 0; q < U; q++) {
        const uint32_t l = q * B + threadIdx.x;
        x[q] = ld_buf(in0, l >= lb0 && l < lb1 ? 16 * (l - lb0 + du0) : kOob);
      }
      if (two) {
        const rsrc_t in1 = make_rsrc(payload + r1.pay_off, 16 * (r1.len >> 4));
        const rsrc_t out1 = make_rsrc(dst + r1.dst_off, 16 * (r1.len >> 4));
        u32x4 y[U];
#pragma unroll
        for (int q = 0; q < U; q++) {
          const uint32_t l = q * B + threadIdx.x;
          y[q] = ld_buf(in1, l >= lb1 ? 16 * (l - lb1) : kOob);
        }
#pragma unroll
        for (int q = 0; q < U; q++) {
          const uint32_t l = q * B + threadIdx.x;
          st_buf(y[q], out1, l >= lb1 ? 16 * (l - lb1) : kOob);
          x[q] |= y[q];
        }
      }
      u64 t0[2] = {0, 0}, t1[2] = {0, 0};
#pragma unroll
      for (int q = 0; q < U; q++) {
        const uint32_t l = q * B + threadIdx.x;
        st_buf(x[q], out0, l >= lb0 && l < lb1 ? 16 * (l - lb0 + du0) : kOob);
        if (l >= lb1) acc4(x[q], 4 * (l - lb1), t1[0], t1[1]);  // zeros add nothing
        else if (l >= lb0) acc4(x[q], 4 * (l - lb0 + du0), t0[0], t0[1]);
      }
      unpack_tile_tail(r0, lb0, du0, T, B, payload, dst, t0);
      if (two) unpack_tile_tail(r1, lb1, 0, T, B, payload, dst, t1);
      block_sum<B, 2>(t0, lds, parity);
      parity ^= 1;
      if (threadIdx.x == 0) add_sum(acc_out + acc_index(wk, r0.c, du0 / wk.sl_vec), t0[0], t0[1]);
      if (two) {  // the second unit starts inside the tile: its slice 0
        block_sum<B, 2>(t1, lds, parity);
        parity ^= 1;
        if (threadIdx.x == 0) add_sum(acc_out + acc_index(wk, r1.c, 0), t1[0], t1[1]);
      }
      continue;
    }
    // Three or more units (short entries): one pass per unit.
    for (u64 u = u0; u < a.n_units; u++) {
      const PlainUnit r = a.units[u];
      const u64 dv = r.dst_off >> 4;
      if (dv >= v_end) break;
      const uint32_t lb = dv > v_blk ? uint32_t(dv - v_blk) : 0u;
      const uint32_t du = v_blk > dv ? uint32_t(v_blk - dv) : 0u;
      const rsrc_t in = make_rsrc(payload + r.pay_off, 16 * (r.len >> 4));
      const rsrc_t out = make_rsrc(dst + r.dst_off, 16 * (r.len >> 4));
      u32x4 x[U];
#pragma unroll
      for (int q = 0; q < U; q++) {
        const uint32_t l = q * B + threadIdx.x;
        x[q] = ld_buf(in, l >= lb ? 16 * (l - lb + du) : kOob);  // zeros past the data
      }
      u64 t[2] = {0, 0};
#pragma unroll
      for (int q = 0; q < U; q++) {
        const uint32_t l = q * B + threadIdx.x;
        st_buf(x[q], out, l >= lb ? 16 * (l - lb + du) : kOob);
        if (l >= lb) acc4(x[q], 4 * (l - lb + du), t[0], t[1]);  // zeros add nothing
      }
      unpack_tile_tail(r, lb, du, T, B, payload, dst, t);
      block_sum<B, 2>(t, lds, parity);
      parity ^= 1;
      if (threadIdx.x == 0) add_sum(acc_out + acc_index(wk, r.c, du / wk.sl_vec), t[0], t[1]);
    }
  }
}

// Delta restore in one launch over a list built on the device: workgroup ids
// first walk the listed sent chunks (wp), then the listed bf16 parameter
// chunks (wd), which are re-derived from their master chunks: a master
// chunk re-sent in this list is read from the payload (pay_of: its offset
// there; kNoPayload if it lies past the readable payload), any other from
// the receiver, which this launch does not write there.  So no slice reads
// what another writes, and the whole delta runs as one kernel.  Parameter
// sums go to list position r.c.
template <int B, int U>
__global__ __launch_bounds__(B) void k_unpack_list(const PlainUnit* __restrict__ plain, Walk wp,
                                                   const DerivedUnit* __restrict__ derived, Walk wd,
                                                   uint32_t cvec, const uint8_t* __restrict__ payload,
                                                   uint8_t* __restrict__ dst,
                                                   const uint32_t* __restrict__ bits,
                                                   const u64* __restrict__ pay_of,
                                                   fr_chunk_sum* __restrict__ acc_out) {
  __shared__ u64 lds[2][B / 64][4];
  __shared__ u64 lds2[2][B / 64][2];
  int parity = 0;
  const u64 np = walk_slices(wp), n = np + walk_slices(wd);
  for (u64 g = blockIdx.x; g < n; g += gridDim.x) {
    if (g < np) {
      const u64 e = slot_of(wp, g);
      const PlainUnit r = plain[e >> 32];
      const uint32_t j = uint32_t(e);
      u64 acc[2] = {0, 0};
      if (!plain_slice<B, U, false>(r, j, wp, payload, dst, acc)) continue;
      block_sum<B, 2>(acc, lds2, parity);
      parity ^= 1;
      if (threadIdx.x == 0) add_sum(acc_out + acc_index(wp, r.c, j), acc[0], acc[1]);
    } else {
      const u64 e = slot_of(wd, g - np);
      DerivedUnit r = derived[e >> 32];
      const uint32_t j = uint32_t(e) & ~kSlotDerived;
      // this slice's master chunk m0 + part, and where its bytes are: the
      // slice indexes the group's master bytes from the group's start, so a
      // part read from the payload is addressed from cvec * part vectors
      // before its offset there
      const uint32_t part = j >> wd.spc_shift;
      const u64 m = u64(r.m0) + part;
      const u64 po = ((bits[m >> 5] >> (m & 31)) & 1u) ? pay_of[m] : kNoPayload;
      const uint8_t* msrc = dst;
      if (po != kNoPayload) {
        msrc = payload;
        r.m_pay_off = po - u64(part) * cvec * 16;
      }
      u64 acc[4] = {0, 0, 0, 0};
      uint32_t got = 0;
      if (!derived_slice<B, U, false, false>(r, j, wd, cvec, msrc, dst, acc, got)) continue;
      block_sum<B, 4>(acc, lds, parity);
      parity ^= 1;
      if (threadIdx.x == 0)
        add_sum(acc_out + ((u64(r.c) << wd.g_shift) + (j >> (kAccSlicesShift + 1))), acc[2], acc[3]);
    }
  }
}

// ---------------------------------------------------------------- verify

// flags[c] <- 1 when any slice of chunk c differs (flags zeroed); with kSums
// the sums of both arenas go to acc_a / acc_b (zeroed).
template <int B, int U, bool kSums, bool kBuf>
__global__ __launch_bounds__(B) void k_verify(const SrcUnit* __restrict__ units, Walk wk,
                                              const uint8_t* __restrict__ a,
                                              const uint8_t* __restrict__ b,
                                              uint32_t* __restrict__ flags,
                                              fr_chunk_sum* __restrict__ acc_a,
                                              fr_chunk_sum* __restrict__ acc_b) {
  __shared__ u64 lds[2][B / 64][4];
  int parity = 0;
  const u64 n_slices = walk_slices(wk);
  for (u64 g = blockIdx.x; g < n_slices; g += gridDim.x) {
    const u64 e = slot_of(wk, g);
    const SrcUnit r = units[e >> 32];
    const uint32_t c = r.c, j = uint32_t(e);
    const uint32_t nvec = r.len >> 4, tail = r.len & 15;
    const uint32_t endv = nvec + (tail ? 1u : 0u);
    const uint32_t lead_v = lead_vectors(wk, r.lead, r.plead);  // as in k_pack
    const uint32_t v0 = j * wk.sl_vec - lead_v;
    if (j * wk.sl_vec >= endv + lead_v) continue;
    const bool last = (j + 1) * wk.sl_vec >= endv + (wk.absorb ? 0u : lead_v);
    const uint32_t n = last && wk.absorb ? endv - v0 : wk.sl_vec;
    const u32x4* pa = reinterpret_cast<const u32x4*>(a + r.src_off);
    const u32x4* pb = reinterpret_cast<const u32x4*>(b + r.src_off);
    u64 acc[4] = {0, 0, 0, 0};
    uint32_t diff = 0;
    u32x4 xa[U], xb[U];
    load_slice<B, U, kBuf>(xa, pa, nvec, v0, wk.sl_vec);
    load_slice<B, U, kBuf>(xb, pb, nvec, v0, wk.sl_vec);
#pragma unroll
    for (int q = 0; q < U; q++) {
      const uint32_t l = q * B + threadIdx.x, v = v0 + l;
      if (l < wk.sl_vec && v < nvec) {
        const u32x4 x = xa[q] ^ xb[q];
        diff |= x.x | x.y | x.z | x.w;
        if (kSums) {
          acc4(xa[q], 4 * v, acc[0], acc[1]);
          acc4(xb[q], 4 * v, acc[2], acc[3]);
        }
      }
    }
    for (uint32_t l = wk.sl_vec + threadIdx.x; l < n; l += B) {  // an absorbing last slice
      const uint32_t v = v0 + l;
      if (v < nvec) {
        const u32x4 ya = ld_nt(pa + v), yb = ld_nt(pb + v);
        const u32x4 x = ya ^ yb;
        diff |= x.x | x.y | x.z | x.w;
        if (kSums) {
          acc4(ya, 4 * v, acc[0], acc[1]);
          acc4(yb, 4 * v, acc[2], acc[3]);
        }
      }
    }
    if (tail && nvec - v0 < n && threadIdx.x == (nvec - v0) % B) {
      const u32x4 ta = load_tail(reinterpret_cast<const uint8_t*>(pa + nvec), tail);
      const u32x4 tb = load_tail(reinterpret_cast<const uint8_t*>(pb + nvec), tail);
      const u32x4 x = ta ^ tb;
      diff |= x.x | x.y | x.z | x.w;
      if (kSums) {
        acc4(ta, 4 * nvec, acc[0], acc[1]);
        acc4(tb, 4 * nvec, acc[2], acc[3]);
      }
    }
    // Any lane of the wave that differs marks the chunk; the store is
    // idempotent, so several waves or slices may make it.
    if (__ballot(diff != 0) != 0 && (threadIdx.x & 63) == 0) flags[c] = 1u;
    if (kSums) {
      block_sum<B, 4>(acc, lds, parity);
      parity ^= 1;
      if (threadIdx.x == 0) {
        const u64 i = acc_index(wk, c, j);
        add_sum(acc_a + i, acc[0], acc[1]);
        add_sum(acc_b + i, acc[2], acc[3]);
      }
    }
  }
}

// -------------------------------------------------------------- finalize

// One lane per chunk.  Modes:
//   kFold:    sums[c] = sum of its G accumulators              (pack, checksum)
//   kCompare: bit c = (sum of its accumulators != sent[c])       (unpack)
//   kFlags:   bit c = (flags[c] != 0); optional folds of two
//             accumulator sets into sums_a / sums_b             (verify)
// Bitmap words are written whole from wave ballots (lanes 0 and 32 each own
// one 32-bit word), so the bitmap needs no clearing.  The count is summed
// per workgroup and added with one atomic per workgroup with a set bit
// (one per wave serialises on the counter when many chunks differ: 30 us
// for 4,096 flipped chunks of the 8B share).
enum FinalMode { kFold = 0, kCompare = 1, kFlags = 2 };

struct FinalArgs {
  const fr_chunk_sum* acc;  // accumulators (A for kFlags)
  const fr_chunk_sum* acc_b;
  const fr_chunk_sum* sent;
  const uint32_t* flags;    // kFlags: the compare's flags; kCompare: NULL, or chunks to flag anyway
  fr_chunk_sum* out;  // sums (A for kFlags)
  fr_chunk_sum* out_b;
  uint32_t* bitmap;
  u64* count;
  uint32_t n_chunks;  // bitmap bits written (ceil(n_chunks / 32) words)
  uint32_t g_shift;
  const u64* live;    // NULL, or a device count: positions from *live on are not chunks (bit 0, no sums)
};

__device__ __forceinline__ fr_chunk_sum fold(const fr_chunk_sum* acc, u64 c, uint32_t g_shift) {
  u64 s = 0, ws = 0;
  const u64 first = c << g_shift;
  for (u64 i = first; i < first + (u64(1) << g_shift); i++) {
    s += acc[i].sum;
    ws += acc[i].wsum;
  }
  return fr_chunk_sum{s, ws};
}

constexpr int kFinalThreads = 1024;

template <int kMode>
__global__ __launch_bounds__(kFinalThreads) void k_finalize(FinalArgs f) {
  __shared__ u64 wave_count[kFinalThreads / 64];
  const uint32_t lane = threadIdx.x & 63;
  const u64 stride = u64(gridDim.x) * blockDim.x;
  u64 count = 0;  // set bits seen by this wave (uniform)
  u64 n_live = f.n_chunks;
  if (f.live && *f.live < n_live) n_live = *f.live;
  for (u64 base = u64(blockIdx.x) * blockDim.x + (threadIdx.x & ~63u); base < f.n_chunks;
       base += stride) {
    const u64 c = base + lane;
    const bool live = c < n_live;
    bool bit = false;
    if (kMode == kFold) {
      if (live) f.out[c] = fold(f.acc, c, f.g_shift);
      continue;
    }
    if (kMode == kCompare && live) {
      const fr_chunk_sum got = fold(f.acc, c, f.g_shift);
      bit = got.sum != f.sent[c].sum || got.wsum != f.sent[c].wsum || (f.flags && f.flags[c]);
    }
    if (kMode == kFlags && live) {
      bit = f.flags[c] != 0;
      if (f.out) {
        f.out[c] = fold(f.acc, c, f.g_shift);
        f.out_b[c] = fold(f.acc_b, c, f.g_shift);
      }
    }
    const u64 mask = __ballot(bit);
    const u64 w = base >> 5;  // base is a multiple of 64: two words per wave
    if (lane == 0) f.bitmap[w] = uint32_t(mask);
    if (lane == 32 && base + 32 < f.n_chunks) f.bitmap[w + 1] = uint32_t(mask >> 32);
    count += u64(__popcll(mask));
  }
  if (kMode == kFold) return;  // uniform over the grid
  if (lane == 0) wave_count[threadIdx.x >> 6] = count;
  __syncthreads();
  if (threadIdx.x == 0) {
    u64 t = 0;
#pragma unroll
    for (int i = 0; i < kFinalThreads / 64; i++) t += wave_count[i];
    if (t) atomicAdd(f.count, t);
  }
}

// ----------------------------------------------------------- delta lists
//
// A delta call's list of chunks, given as a bitmap over the plan's chunk
// ids (bit c set: chunk c is listed; list positions follow chunk order),
// becomes the call's unit records on the device, so a repair from the
// compare's bitmap needs no host round trip.  In the delta payload a sent
// chunk that continues the previous sent chunk of its entry follows it, any
// other starts at the next multiple of the segment alignment A.  Where a
// chunk lands depends on every chunk before it, but each one acts on the
// running payload end x as x -> x + len (continuing) or x -> align_A(x) +
// len, and such maps compose within the family {x -> x + q} u
// {x -> align_A(x + p) + q}, because align_A(align_A(z) + w) = align_A(z) +
// align_A(w) for w >= 0: a prefix scan over the chunks places them all.
// One lane per chunk id, blocks of kListBlock ids:
//   k_list_blocks  each block's composed map and counts (a scan over its
//                  lanes with cross-lane shuffles, then LDS over its waves);
//   k_list_scan    one workgroup: every block's payload end and counts
//                  before it, and the totals;
//   k_list_build   each lane places its chunk from its block's start and the
//                  scan within the block, and writes its unit records.

__device__ __forceinline__ u64 align_a(u64 x, u64 a) { return (x + a - 1) & ~(a - 1); }

__device__ __forceinline__ DeltaAgg delta_identity() { return DeltaAgg{0, 0, 0, 0, 0, 0}; }

// g after f.
__device__ __forceinline__ DeltaAgg delta_then(const DeltaAgg& f, const DeltaAgg& g, u64 A) {
  DeltaAgg h;
  h.ns = f.ns + g.ns;
  h.nd = f.nd + g.nd;
  h.pad_ = 0;
  if (!g.has) {
    h.has = f.has;
    h.p = f.p;
    h.q = f.q + g.q;
  } else if (!f.has) {
    h.has = 1;
    h.p = f.q + g.p;
    h.q = g.q;
  } else {
    h.has = 1;
    h.p = f.p;
    h.q = align_a(f.q + g.p, A) + g.q;
  }
  return h;
}

__device__ __forceinline__ u64 delta_apply(const DeltaAgg& f, u64 x, u64 A) {
  return f.has ? align_a(x + f.p, A) + f.q : x + f.q;
}

__device__ __forceinline__ DeltaAgg shfl_up_agg(const DeltaAgg& a, uint32_t d) {
  DeltaAgg o;
  o.ns = uint32_t(__shfl_up(int(a.ns), d, 64));
  o.nd = uint32_t(__shfl_up(int(a.nd), d, 64));
  o.has = uint32_t(__shfl_up(int(a.has), d, 64));
  o.pad_ = 0;
  o.p = u64(__shfl_up((long long)a.p, d, 64));
  o.q = u64(__shfl_up((long long)a.q, d, 64));
  return o;
}

__device__ __forceinline__ bool listed(const uint32_t* bits, u64 c, u64 n_chunks) {
  return c < n_chunks && ((bits[c >> 5] >> (c & 31)) & 1u);
}

// Lane c's chunk: its element of the scan and its location (valid if listed).
struct ListLane {
  bool on;        // listed
  bool cont;      // sent, continuing the previous listed chunk of its entry
  bool next_cont; // sent, and the next chunk of its entry is listed
  ChunkLoc loc;
  DeltaAgg e;
};

__device__ __forceinline__ ListLane list_lane(const DeltaBuild& b, u64 c) {
  ListLane l;
  l.on = listed(b.bits, c, b.n_chunks);
  l.cont = l.next_cont = false;
  l.e = delta_identity();
  if (!l.on) return l;
  l.loc = b.loc[c];
  if (l.loc.flags & kLocDerived) {
    l.e.nd = 1;
    return l;
  }
  l.cont = !(l.loc.flags & kLocFirst) && listed(b.bits, c - 1, b.n_chunks);
  l.next_cont = !(l.loc.flags & kLocLast) && listed(b.bits, c + 1, b.n_chunks);
  l.e.ns = 1;
  l.e.has = l.cont ? 0u : 1u;
  l.e.q = l.loc.len;
  return l;
}

// Scan of `e` over the kThreads lanes of a workgroup (cross-lane shuffles
// within each wave, then the wave totals through LDS): `excl` receives the
// lane's exclusive prefix, and the return value is the workgroup's total.
// Every lane must call it.
template <int kThreads>
__device__ __forceinline__ DeltaAgg block_scan(DeltaAgg e, u64 A, DeltaAgg& excl) {
  __shared__ DeltaAgg wave_total[kThreads / 64];
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  DeltaAgg inc = e;
  for (uint32_t d = 1; d < 64; d <<= 1) {
    const DeltaAgg o = shfl_up_agg(inc, d);
    if (lane >= d) inc = delta_then(o, inc, A);
  }
  if (lane == 63) wave_total[wave] = inc;
  // every lane takes part in the shuffle (a lane reading an inactive lane
  // gets nothing), lane 0 then drops what it read
  const DeltaAgg prev = shfl_up_agg(inc, 1);
  const DeltaAgg wexcl = lane ? prev : delta_identity();
  __syncthreads();
  DeltaAgg before = delta_identity();  // the waves before this one
  for (uint32_t w = 0; w < wave; w++) before = delta_then(before, wave_total[w], A);
  excl = delta_then(before, wexcl, A);
  DeltaAgg total = before;
  for (uint32_t w = wave; w < kThreads / 64; w++) total = delta_then(total, wave_total[w], A);
  return total;
}

__global__ __launch_bounds__(kListBlock) void k_list_blocks(DeltaBuild b) {
  const u64 c = u64(blockIdx.x) * kListBlock + threadIdx.x;
  const ListLane l = list_lane(b, c);
  DeltaAgg excl;
  const DeltaAgg total = block_scan<kListBlock>(l.e, b.seg, excl);
  if (threadIdx.x == 0) b.agg[blockIdx.x] = total;
}

constexpr int kScanThreads = 1024;

// Thread i composes blocks [i k, (i + 1) k); a scan over the threads gives
// each thread the map of everything before its blocks; it then walks its
// blocks again with the running payload end.
__global__ __launch_bounds__(kScanThreads) void k_list_scan(DeltaBuild b, u64 n_blocks) {
  const uint32_t i = threadIdx.x;
  const u64 k = (n_blocks + kScanThreads - 1) / kScanThreads;
  const u64 w0 = u64(i) * k < n_blocks ? u64(i) * k : n_blocks;
  const u64 w1 = w0 + k < n_blocks ? w0 + k : n_blocks;
  const u64 A = b.seg;
  DeltaAgg a = delta_identity();
  for (u64 w = w0; w < w1; w++) a = delta_then(a, b.agg[w], A);
  DeltaAgg before;
  const DeltaAgg all = block_scan<kScanThreads>(a, A, before);
  u64 x = delta_apply(before, 0, A);
  uint32_t ns = before.ns, nd = before.nd;
  for (u64 w = w0; w < w1; w++) {
    b.pre[w] = DeltaPre{x, ns, nd};
    const DeltaAgg g = b.agg[w];
    x = delta_apply(g, x, A);
    ns += g.ns;
    nd += g.nd;
  }
  if (i == 0) {
    const u64 end = delta_apply(all, 0, A);
    b.counts[kDeltaIds] = u64(all.ns) + all.nd;
    b.counts[kDeltaSent] = all.ns;
    b.counts[kDeltaDerived] = all.nd;
    b.counts[kDeltaEnd] = end;
    if (b.user_counts) {
      b.user_counts[0] = u64(all.ns) + all.nd;
      b.user_counts[1] = align_a(end, 16);
    }
    if (b.zero_word) *b.zero_word = 0;
  }
}

template <bool kForPack>
__global__ __launch_bounds__(kListBlock) void k_list_build(DeltaBuild b) {
  const u64 c = u64(blockIdx.x) * kListBlock + threadIdx.x;
  const ListLane l = list_lane(b, c);
  DeltaAgg excl;
  (void)block_scan<kListBlock>(l.e, b.seg, excl);
  if (!l.on) return;
  const DeltaPre pre = b.pre[blockIdx.x];
  const u64 A = b.seg;
  const uint32_t pos = pre.ns + pre.nd + excl.ns + excl.nd;  // list position
  for (uint32_t a = 0; a < (1u << b.acc_shift); a++)
    b.acc[(u64(pos) << b.acc_shift) + a] = fr_chunk_sum{0, 0};
  const ChunkLoc& r = l.loc;
  if (r.flags & kLocDerived) {
    if (kForPack) {
      b.src_units[pos] = SrcUnit{r.src_off, kNoPayload, r.len, pos, 0, uint16_t(r.src_off % kLeadMod), 0};
    } else {
      // re-derived from its master chunks: m_pay_off is their receiver offset,
      // and a master chunk re-sent in this list is read from the payload
      // instead (the unpack finds its offset in pay_of)
      b.derived[pre.nd + excl.nd] =
          DerivedUnit{r.m_dst_off, r.m_dst_off, r.dst_off, r.len, b.m0[c], pos, 0};
      b.bad[pos] = 0;
    }
    return;
  }
  const u64 x = delta_apply(excl, pre.end, A);  // the payload end before this chunk
  const u64 pay = l.cont ? x : align_a(x, A);
  const u64 end = pay + r.len;
  if (kForPack) {
    // zero gap up to the next sent chunk: none after the last one or before
    // a continuing one, else up to the next segment boundary
    const u64 gap =
        (end == b.counts[kDeltaEnd] || l.next_cont) ? 0 : align_a(end, A) - align_a(end, 16);
    const bool fits = align_a(end, 16) + gap <= b.payload_limit;  // never false for a checked cap
    b.src_units[pos] = SrcUnit{r.src_off, fits ? pay : kNoPayload, r.len, pos,
                               fits ? uint32_t(gap >> 4) : 0u, uint16_t(r.src_off % kLeadMod),
                               uint16_t(pay % kLeadMod)};
  } else {
    // a chunk past the readable payload is neither read nor written, and flagged
    const bool readable = align_a(end, 16) <= b.payload_limit;
    b.plain[pre.ns + excl.ns] =
        PlainUnit{readable ? pay : 0, r.dst_off, readable ? r.len : 0u, pos, uint32_t(pay % kLeadMod),
                  uint32_t(r.dst_off % kLeadMod)};
    b.bad[pos] = readable ? 0u : 1u;
    b.pay_of[c] = readable ? pay : kNoPayload;
  }
}

__global__ __launch_bounds__(256) void k_ids_to_bits(const uint32_t* __restrict__ ids, u64 n,
                                                     uint32_t* __restrict__ bits) {
  const u64 i = u64(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) atomicOr(bits + (ids[i] >> 5), 1u << (ids[i] & 31u));
}

// ------------------------------------------------------------- utilities

// Expands a slot table from runs (plan creation).  Thread o writes entry o
// of the XCD-major image, which holds slot g = (o mod stride) * 8 +
// o / stride, so consecutive threads store consecutive words; slot g belongs
// to the last run whose first slot is <= g (binary search: first[0] = 0 <=
// g < n = first[n_runs], and no run is empty).
__global__ __launch_bounds__(256) void k_expand_slots(const u64* __restrict__ first,
                                                      const u64* __restrict__ base, u64 n_runs,
                                                      u64 n, u64 stride, u64* __restrict__ out) {
  const u64 total = 8 * stride, step = u64(gridDim.x) * blockDim.x;
  for (u64 o = u64(blockIdx.x) * blockDim.x + threadIdx.x; o < total; o += step) {
    const u64 g = (o % stride) * 8 + o / stride;
    u64 v = 0;
    if (g < n) {
      u64 lo = 0, hi = n_runs;  // first[lo] <= g < first[hi]
      while (hi - lo > 1) {
        const u64 mid = lo + (hi - lo) / 2;
        if (first[mid] <= g) lo = mid;
        else hi = mid;
      }
      v = base[lo] | (g - first[lo]);
    }
    out[o] = v;
  }
}

// Clears up to four regions of 32-bit words (a kernel rather than a memset
// so that an operation is made of kernel launches only).
struct ZeroList {
  uint32_t* p[4];
  u64 words[4];
};

__global__ __launch_bounds__(256) void k_zero(ZeroList z) {
  const u64 stride = u64(gridDim.x) * blockDim.x;
#pragma unroll
  for (int r = 0; r < 4; r++) {
    uint32_t* p = z.p[r];
    for (u64 i = u64(blockIdx.x) * blockDim.x + threadIdx.x; i < z.words[r]; i += stride) p[i] = 0;
  }
}

struct Zeroes {
  ZeroList z{};
  int n = 0;
  u64 total = 0;
  void add(void* p, u64 bytes) {
    if (!p || bytes == 0) return;
    z.p[n] = static_cast<uint32_t*>(p);
    z.words[n] = bytes / 4;
    total += bytes / 4;
    n++;
  }
  int launch(hipStream_t st) {
    if (n == 0) return 0;
    const u64 want = (total + 255) / 256;
    const uint32_t blocks = uint32_t(want < 2048 ? (want ? want : 1) : 2048);
    hipLaunchKernelGGL(k_zero, dim3(blocks), dim3(256), 0, st, z);
    return int(hipGetLastError());
  }
};

// Workgroups per launch: one per slice up to the configured cap and the
// hardware limit of 2^32 work-items per grid; beyond that, grid-stride.
template <int B>
inline uint32_t grid_for(u64 units, const LaunchCfg& cfg) {
  u64 cap = (u64(1) << 31) / B;
  if (cfg.max_grid && cfg.max_grid < cap) cap = cfg.max_grid;
  return uint32_t(units < cap ? units : cap);
}

// A walk over a list built on the device covers the list's largest possible
// length; its grid is capped (workgroups then loop), so that a short list
// does not pay for the dispatch of a grid sized for the longest.
template <int B>
inline uint32_t grid_of(const Walk& wk, const LaunchCfg& cfg) {
  uint32_t g = grid_for<B>(wk.n_slices, cfg);
  if (wk.count && cfg.delta_grid && g > cfg.delta_grid) g = cfg.delta_grid;
  return g;
}

// Slice geometry for chunks of C bytes and a tile of `tile_bytes`, walked by
// the slot table `t` (built for that slice size).
inline Walk walk_for(uint64_t C, uint32_t tile_bytes, const SlotTable& t) {
  const uint64_t sl = C < tile_bytes ? C : tile_bytes;
  uint32_t sh = 0;
  while ((sl << sh) < C) sh++;
  Walk w;
  w.slots = reinterpret_cast<const u64*>(t.d);
  w.n_slices = t.n;
  w.stride = t.stride;
  w.imp_shift = t.implicit_shift;
  w.sl_vec = uint32_t(sl >> 4);
  w.line = t.shift;
  w.absorb = t.absorb;
  w.count = reinterpret_cast<const u64*>(t.count);
  w.spc_shift = sh;
  w.g_shift = sh > kAccSlicesShift ? sh - kAccSlicesShift : 0;
  return w;
}

inline int launch_finalize(int mode, const FinalArgs& f, hipStream_t st) {
  if (f.n_chunks == 0) return 0;
  const u64 waves = (u64(f.n_chunks) + 63) / 64;
  const u64 want = (waves + kFinalThreads / 64 - 1) / (kFinalThreads / 64);
  const dim3 grid(uint32_t(want < 2048 ? want : 2048)), block(kFinalThreads);
  if (mode == kFold) hipLaunchKernelGGL(k_finalize<kFold>, grid, block, 0, st, f);
  else if (mode == kCompare) hipLaunchKernelGGL(k_finalize<kCompare>, grid, block, 0, st, f);
  else hipLaunchKernelGGL(k_finalize<kFlags>, grid, block, 0, st, f);
  return int(hipGetLastError());
}

// Launch configurations: B threads x U vectors per slice.
enum Tile {
  T256x1 = 0, T512x1 = 1, T256x2 = 2, T256x4 = 3, T64x4 = 4, T128x2 = 5,
  T64x2 = 6, T64x1 = 7, T128x1 = 8, T128x4 = 9, T64x8 = 10
};

template <int B, int U>
int pack_impl(bool store, const SrcUnit* units, const SlotTable& slots, uint32_t n_chunks,
              uint64_t C, const void* src, void* payload, fr_chunk_sum* sums, const Scratch& scr,
              const LaunchCfg& cfg, hipStream_t st) {
  if (n_chunks == 0) return 0;
  const Walk wk = walk_for(C, B * U * 16, slots);
  const u64 n_acc = u64(n_chunks) << wk.g_shift;
  Zeroes z;
  if (!wk.count)  // a list built on the device: its builder cleared the accumulators
    z.add(scr.acc, n_acc * sizeof(fr_chunk_sum));
  int e = z.launch(st);
  if (e) return e;
  const auto* s = static_cast<const uint8_t*>(src);
  auto* p = static_cast<uint8_t*>(payload);
  const dim3 grid(grid_of<B>(wk, cfg));
  if (store && cfg.buf_pack)
    hipLaunchKernelGGL((k_pack<B, U, true, true>), grid, dim3(B), 0, st, units, wk, s, p, scr.acc);
  else if (store)
    hipLaunchKernelGGL((k_pack<B, U, true, false>), grid, dim3(B), 0, st, units, wk, s, p, scr.acc);
  else if (cfg.buf_checksum)
    hipLaunchKernelGGL((k_pack<B, U, false, true>), grid, dim3(B), 0, st, units, wk, s, p, scr.acc);
  else
    hipLaunchKernelGGL((k_pack<B, U, false, false>), grid, dim3(B), 0, st, units, wk, s, p, scr.acc);
  e = int(hipGetLastError());
  if (e) return e;
  FinalArgs f{};
  f.acc = scr.acc;
  f.out = sums;
  f.n_chunks = n_chunks;
  f.g_shift = wk.g_shift;
  f.live = wk.count;  // a list built on the device: its length
  return launch_finalize(kFold, f, st);
}

template <int B, int U>
int pack_blocks_impl(const SrcUnit* units, const PackBlocks& pb, uint32_t n_chunks, uint64_t C,
                     const void* src, void* payload, fr_chunk_sum* sums, const Scratch& scr,
                     const LaunchCfg& cfg, hipStream_t st) {
  if (n_chunks == 0) return 0;
  const Walk wk = walk_for(C, B * U * 16, pb.extra);
  Zeroes z;
  z.add(scr.acc, (u64(n_chunks) << wk.g_shift) * sizeof(fr_chunk_sum));
  int e = z.launch(st);
  if (e) return e;
  PackBlocksArgs a;
  a.pay_units = pb.units;
  a.first = pb.first;
  a.n_units = pb.n_units;
  a.n_blocks = pb.n_blocks;
  a.stride = pb.stride;
  a.pay_vecs = pb.pay_vecs;
  const auto* s = static_cast<const uint8_t*>(src);
  auto* p = static_cast<uint8_t*>(payload);
  if (a.n_blocks) {
    hipLaunchKernelGGL((k_pack_blocks<B, U>), dim3(grid_for<B>(a.n_blocks, cfg)), dim3(B), 0, st, a,
                       wk, s, p, scr.acc);
    e = int(hipGetLastError());
    if (e) return e;
  }
  if (wk.n_slices) {
    hipLaunchKernelGGL((k_pack<B, U, true, true>), dim3(grid_for<B>(wk.n_slices, cfg)), dim3(B), 0,
                       st, units, wk, s, p, scr.acc);
    e = int(hipGetLastError());
    if (e) return e;
  }
  FinalArgs f{};
  f.acc = scr.acc;
  f.out = sums;
  f.n_chunks = n_chunks;
  f.g_shift = wk.g_shift;
  return launch_finalize(kFold, f, st);
}

template <int B, int U>
int unpack_impl(const UnpackArgs& u, const LaunchCfg& cfg, hipStream_t st) {
  const Walk wk = walk_for(u.C, B * U * 16, u.slots);
  const u64 n_acc = u64(u.n_chunks) << wk.g_shift;
  Zeroes z;
  z.add(u.scratch.acc, n_acc * sizeof(fr_chunk_sum));
  z.add(u.n_bad, 8);
  int e = z.launch(st);
  if (e || u.n_chunks == 0) return e;
  if (wk.n_slices) {
    if (cfg.buf_unpack)
      hipLaunchKernelGGL((k_unpack<B, U, true>), dim3(grid_for<B>(wk.n_slices, cfg)), dim3(B), 0, st,
                         u.derived, u.plain, wk, uint32_t(u.C >> 4),
                         static_cast<const uint8_t*>(u.payload), static_cast<uint8_t*>(u.dst),
                         u.scratch.acc);
    else
      hipLaunchKernelGGL((k_unpack<B, U, false>), dim3(grid_for<B>(wk.n_slices, cfg)), dim3(B), 0, st,
                         u.derived, u.plain, wk, uint32_t(u.C >> 4),
                         static_cast<const uint8_t*>(u.payload), static_cast<uint8_t*>(u.dst),
                         u.scratch.acc);
    e = int(hipGetLastError());
    if (e) return e;
  }
  FinalArgs f{};
  f.acc = u.scratch.acc;
  f.sent = u.sums;
  f.bitmap = u.bitmap;
  f.count = reinterpret_cast<u64*>(u.n_bad);
  f.n_chunks = u.n_chunks;
  f.g_shift = wk.g_shift;
  return launch_finalize(kCompare, f, st);
}

template <int B, int U>
int unpack_blocks_impl(const UnpackArgs& u, const UnpackBlocks& ub, const LaunchCfg& cfg,
                       hipStream_t st) {
  const Walk wk = walk_for(u.C, B * U * 16, ub.derived);
  const u64 n_acc = u64(u.n_chunks) << wk.g_shift;
  Zeroes z;
  z.add(u.scratch.acc, n_acc * sizeof(fr_chunk_sum));
  z.add(u.n_bad, 8);
  int e = z.launch(st);
  if (e || u.n_chunks == 0) return e;
  const auto* pay = static_cast<const uint8_t*>(u.payload);
  auto* dst = static_cast<uint8_t*>(u.dst);
  if (ub.n_blocks) {
    UnpackBlocksArgs a;
    a.units = ub.units;
    a.blocks = reinterpret_cast<const u64*>(ub.blocks);
    a.n_units = ub.n_units;
    a.n_blocks = ub.n_blocks;
    a.stride = ub.stride;
    hipLaunchKernelGGL((k_unpack_blocks<B, U>), dim3(grid_for<B>(ub.n_blocks, cfg)), dim3(B), 0, st,
                       a, wk, pay, dst, u.scratch.acc);
    e = int(hipGetLastError());
    if (e) return e;
  }
  if (wk.n_slices) {  // the derived groups
    hipLaunchKernelGGL((k_unpack<B, U, false>), dim3(grid_for<B>(wk.n_slices, cfg)), dim3(B), 0, st,
                       u.derived, u.plain, wk, uint32_t(u.C >> 4), pay, dst, u.scratch.acc);
    e = int(hipGetLastError());
    if (e) return e;
  }
  FinalArgs f{};
  f.acc = u.scratch.acc;
  f.sent = u.sums;
  f.bitmap = u.bitmap;
  f.count = reinterpret_cast<u64*>(u.n_bad);
  f.n_chunks = u.n_chunks;
  f.g_shift = wk.g_shift;
  return launch_finalize(kCompare, f, st);
}

template <int B, int U>
int unpack_delta_impl(const UnpackDeltaArgs& u, const LaunchCfg& cfg, hipStream_t st) {
  const Walk wd = walk_for(u.C, B * U * 16, u.derived_slots);
  const Walk wp = walk_for(u.C, B * U * 16, u.plain_slots);
  const u64 n_acc = u64(u.n_ids) << wp.g_shift;
  Zeroes z;
  if (!u.live) {  // else the list's builder cleared the accumulators and n_bad
    z.add(u.scratch.acc, n_acc * sizeof(fr_chunk_sum));
    z.add(u.n_bad, 8);
  }
  int e = z.launch(st);
  if (e || u.n_ids == 0) return e;
  const uint32_t cvec = uint32_t(u.C >> 4);
  if (wp.n_slices + wd.n_slices) {  // sent and derived chunks in one launch
    Walk both = wp;
    both.n_slices = wp.n_slices + wd.n_slices;
    hipLaunchKernelGGL((k_unpack_list<B, U>), dim3(grid_of<B>(both, cfg)), dim3(B), 0, st, u.plain,
                       wp, u.derived, wd, cvec, static_cast<const uint8_t*>(u.payload),
                       static_cast<uint8_t*>(u.dst), u.bits, reinterpret_cast<const u64*>(u.pay_of),
                       u.scratch.acc);
    e = int(hipGetLastError());
    if (e) return e;
  }
  FinalArgs f{};
  f.acc = u.scratch.acc;
  f.sent = u.sums;
  f.bitmap = u.bitmap;
  f.count = reinterpret_cast<u64*>(u.n_bad);
  f.n_chunks = u.n_ids;
  f.g_shift = wp.g_shift;
  f.live = reinterpret_cast<const u64*>(u.live);
  f.flags = u.bad;
  return launch_finalize(kCompare, f, st);
}

template <int B, int U>
int verify_impl(const SrcUnit* units, const SlotTable& slots, uint32_t n_chunks, uint64_t C,
                const void* a, const void* b, uint32_t* bitmap, uint64_t* n_diff,
                fr_chunk_sum* sums_a, fr_chunk_sum* sums_b, const Scratch& scr,
                const LaunchCfg& cfg, hipStream_t st) {
  const Walk wk = walk_for(C, B * U * 16, slots);
  const u64 n_acc = u64(n_chunks) << wk.g_shift;
  Zeroes z;
  z.add(scr.flags, u64(n_chunks) * 4);
  z.add(n_diff, 8);
  if (sums_a) {
    z.add(scr.acc, n_acc * sizeof(fr_chunk_sum));
    z.add(scr.acc_b, n_acc * sizeof(fr_chunk_sum));
  }
  int e = z.launch(st);
  if (e || n_chunks == 0) return e;
  const auto* pa = static_cast<const uint8_t*>(a);
  const auto* pb = static_cast<const uint8_t*>(b);
  const dim3 grid(grid_for<B>(wk.n_slices, cfg));
  if (sums_a && cfg.buf_verify)
    hipLaunchKernelGGL((k_verify<B, U, true, true>), grid, dim3(B), 0, st, units, wk, pa, pb,
                       scr.flags, scr.acc, scr.acc_b);
  else if (sums_a)
    hipLaunchKernelGGL((k_verify<B, U, true, false>), grid, dim3(B), 0, st, units, wk, pa, pb,
                       scr.flags, scr.acc, scr.acc_b);
  else if (cfg.buf_verify)
    hipLaunchKernelGGL((k_verify<B, U, false, true>), grid, dim3(B), 0, st, units, wk, pa, pb,
                       scr.flags, scr.acc, scr.acc_b);
  else
    hipLaunchKernelGGL((k_verify<B, U, false, false>), grid, dim3(B), 0, st, units, wk, pa, pb,
                       scr.flags, scr.acc, scr.acc_b);
  e = int(hipGetLastError());
  if (e) return e;
  FinalArgs f{};
  f.acc = scr.acc;
  f.acc_b = scr.acc_b;
  f.flags = scr.flags;
  f.out = sums_a;
  f.out_b = sums_b;
  f.bitmap = bitmap;
  f.count = reinterpret_cast<u64*>(n_diff);
  f.n_chunks = n_chunks;
  f.g_shift = wk.g_shift;
  return launch_finalize(kFlags, f, st);
}

#define FR_DISPATCH(tile, fn, ...)                        \
  switch (tile) {                                         \
    case T512x1: return fn<512, 1>(__VA_ARGS__);          \
    case T256x2: return fn<256, 2>(__VA_ARGS__);          \
    case T256x4: return fn<256, 4>(__VA_ARGS__);          \
    case T64x4: return fn<64, 4>(__VA_ARGS__);            \
    case T128x2: return fn<128, 2>(__VA_ARGS__);          \
    case T64x2: return fn<64, 2>(__VA_ARGS__);            \
    case T64x1: return fn<64, 1>(__VA_ARGS__);            \
    case T128x1: return fn<128, 1>(__VA_ARGS__);          \
    case T128x4: return fn<128, 4>(__VA_ARGS__);          \
    case T64x8: return fn<64, 8>(__VA_ARGS__);            \
    default: return fn<256, 1>(__VA_ARGS__);              \
  }

}  // namespace

int launch_expand_slots(const uint64_t* first, const uint64_t* base, uint64_t n_runs, uint64_t n,
                        uint64_t stride, uint64_t* out, void* stream) {
  const u64 total = 8 * stride;
  if (total == 0) return 0;
  const u64 want = (total + 255) / 256;
  const uint32_t blocks = uint32_t(want < 65536 ? want : 65536);
  hipLaunchKernelGGL(k_expand_slots, dim3(blocks), dim3(256), 0, hipStream_t(stream),
                     reinterpret_cast<const u64*>(first), reinterpret_cast<const u64*>(base),
                     u64(n_runs), u64(n), u64(stride), reinterpret_cast<u64*>(out));
  return int(hipGetLastError());
}

int launch_delta_build(const DeltaBuild& b, bool for_pack, void* stream) {
  const hipStream_t st = hipStream_t(stream);
  const u64 n_blocks = (b.n_chunks + kListBlock - 1) / kListBlock;
  const dim3 grid = dim3(uint32_t(n_blocks)), block = dim3(kListBlock);
  if (n_blocks) {
    hipLaunchKernelGGL(k_list_blocks, grid, block, 0, st, b);
    if (const hipError_t e = hipGetLastError()) return int(e);
  }
  hipLaunchKernelGGL(k_list_scan, dim3(1), dim3(kScanThreads), 0, st, b, n_blocks);
  if (const hipError_t e = hipGetLastError()) return int(e);
  if (n_blocks) {
    if (for_pack) hipLaunchKernelGGL(k_list_build<true>, grid, block, 0, st, b);
    else hipLaunchKernelGGL(k_list_build<false>, grid, block, 0, st, b);
  }
  return int(hipGetLastError());
}

int launch_ids_to_bits(const uint32_t* ids, uint64_t n, uint32_t* bits, uint64_t words,
                       void* stream) {
  const hipStream_t st = hipStream_t(stream);
  Zeroes z;
  z.add(bits, words * 4);
  const int e = z.launch(st);
  if (e || n == 0) return e;
  hipLaunchKernelGGL(k_ids_to_bits, dim3(uint32_t((n + 255) / 256)), dim3(256), 0, st, ids, u64(n),
                     bits);
  return int(hipGetLastError());
}

uint32_t tile_bytes(int tile) {
  switch (tile) {
    case T512x1: return 512 * 16;
    case T256x2: return 256 * 2 * 16;
    case T256x4: return 256 * 4 * 16;
    case T64x4: return 64 * 4 * 16;
    case T128x2: return 128 * 2 * 16;
    case T64x2: return 64 * 2 * 16;
    case T64x1: return 64 * 16;
    case T128x1: return 128 * 16;
    case T128x4: return 128 * 4 * 16;
    case T64x8: return 64 * 8 * 16;
    default: return 256 * 16;
  }
}

uint64_t accumulators_per_chunk(uint64_t C, int tile) {
  const Walk w = walk_for(C, tile_bytes(tile), SlotTable{});
  return uint64_t(1) << w.g_shift;
}

int launch_pack(const SrcUnit* units, const SlotTable& slots, uint32_t n_chunks, uint64_t C,
                const void* src, void* payload, fr_chunk_sum* sums, const Scratch& scr,
                const LaunchCfg& cfg, void* stream) {
  FR_DISPATCH(cfg.tile_pack, pack_impl, true, units, slots, n_chunks, C, src, payload, sums, scr,
              cfg, hipStream_t(stream));
}

int launch_pack_blocks(const SrcUnit* units, const PackBlocks& pb, uint32_t n_chunks, uint64_t C,
                       const void* src, void* payload, fr_chunk_sum* sums, const Scratch& scr,
                       const LaunchCfg& cfg, void* stream) {
  FR_DISPATCH(cfg.tile_pack, pack_blocks_impl, units, pb, n_chunks, C, src, payload, sums, scr, cfg,
              hipStream_t(stream));
}

int launch_block_first(const uint64_t* pay_off, uint64_t n_units, uint64_t n_blocks,
                       uint64_t stride, uint32_t block_vecs, uint32_t* out, void* stream) {
  const u64 total = 8 * stride;
  if (total == 0) return 0;
  const u64 want = (total + 255) / 256;
  const uint32_t blocks = uint32_t(want < 65536 ? want : 65536);
  hipLaunchKernelGGL(k_block_first, dim3(blocks), dim3(256), 0, hipStream_t(stream),
                     reinterpret_cast<const u64*>(pay_off), u64(n_units), u64(n_blocks), u64(stride), block_vecs, out);
  return int(hipGetLastError());
}

int launch_checksum(const SrcUnit* units, const SlotTable& slots, uint32_t n_chunks, uint64_t C,
                    const void* base, fr_chunk_sum* sums, const Scratch& scr,
                    const LaunchCfg& cfg, void* stream) {
  FR_DISPATCH(cfg.tile_checksum, pack_impl, false, units, slots, n_chunks, C, base, nullptr, sums,
              scr, cfg, hipStream_t(stream));
}

int launch_unpack(const UnpackArgs& u, const LaunchCfg& cfg, void* stream) {
  FR_DISPATCH(cfg.tile_unpack, unpack_impl, u, cfg, hipStream_t(stream));
}

int launch_unpack_blocks(const UnpackArgs& u, const UnpackBlocks& ub, const LaunchCfg& cfg,
                         void* stream) {
  FR_DISPATCH(cfg.tile_unpack, unpack_blocks_impl, u, ub, cfg, hipStream_t(stream));
}

int launch_unpack_delta(const UnpackDeltaArgs& u, const LaunchCfg& cfg, void* stream) {
  FR_DISPATCH(cfg.tile_unpack, unpack_delta_impl, u, cfg, hipStream_t(stream));
}

int launch_compare_sums(const fr_chunk_sum* a, const fr_chunk_sum* b, uint32_t n_chunks,
                        uint32_t* bitmap, uint64_t* count, void* stream) {
  // the compare finalize with one accumulator per chunk: the first sums
  // folded (as they are) against the second as the sums sent
  const hipStream_t st = hipStream_t(stream);
  Zeroes z;
  z.add(count, sizeof(u64));
  const int e = z.launch(st);
  if (e) return e;
  FinalArgs f{};
  f.acc = a;
  f.sent = b;
  f.bitmap = bitmap;
  f.count = reinterpret_cast<u64*>(count);
  f.n_chunks = n_chunks;
  f.g_shift = 0;
  return launch_finalize(kCompare, f, st);
}

int launch_verify(const SrcUnit* units, const SlotTable& slots, uint32_t n_chunks, uint64_t C,
                  const void* a, const void* b, uint32_t* bitmap, uint64_t* n_diff,
                  fr_chunk_sum* sums_a, fr_chunk_sum* sums_b, const Scratch& scr,
                  const LaunchCfg& cfg, void* stream) {
  FR_DISPATCH(cfg.tile_verify, verify_impl, units, slots, n_chunks, C, a, b, bitmap, n_diff,
              sums_a, sums_b, scr, cfg, hipStream_t(stream));
}

// ------------------------------------------------------- static scratch

// Device memory for the calls that allocate nothing (fr_verify_replicas_noalloc):
// their flags and accumulators live here instead of in the plan's scratch.
// Every GPU the library runs on holds its own copy at its own address until
// the process ends.  In host code `scratch` names a host-side stand-in, not
// device memory: host code uses only the address hipGetSymbolAddress returns
// for the current device, resolved once per device below.
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

int static_scratch_address(int device, void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  if (device < 0 || device >= kMaxDevices) return int(hipErrorInvalidDevice);
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));  // current device's copy
    if (e != hipSuccess) return int(e);
    addr[device] = p;
  }
  *out = addr[device];
  return 0;
}

}  // namespace fr
