// C-ABI entry points of the four operations: synchronous argument checks,
// then stream-ordered kernel launches.  Nothing is enqueued and no output is
// touched unless every check passes.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "fr_internal.h"

namespace fr {
extern thread_local int g_last_hip_error;
}

using namespace fr;

namespace {

struct Region {
  const void* p;
  uint64_t bytes;
};

int device_error(hipError_t e) {
  g_last_hip_error = int(e);
  return FR_E_DEVICE;
}

int check_device_and_stream(const fr_plan* plan, hipStream_t stream) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return device_error(e);
  if (dev != plan->device) return FR_E_DEVICE_MISMATCH;
  if (stream) {
    hipDevice_t sd = -1;
    e = hipStreamGetDevice(hipStream_t(stream), &sd);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return FR_E_INVAL;
    }
    if (int(sd) != plan->device) return FR_E_DEVICE_MISMATCH;
  }
  return FR_OK;
}

// A buffer the kernels will touch: it must be device memory of the plan's
// device, aligned, and lie inside one allocation.  An empty buffer is never
// touched, so any pointer (NULL included) is accepted for it.
int check_buffer(const fr_plan* plan, const void* p, uint64_t bytes, uint64_t align) {
  if (bytes == 0) return FR_OK;
  if (p == nullptr) return FR_E_INVAL;
  if (reinterpret_cast<uintptr_t>(p) % align) return FR_E_ALIGN;
  hipPointerAttribute_t attr{};
  hipError_t e = hipPointerGetAttributes(&attr, p);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return FR_E_INVAL;  // not memory HIP knows about
  }
  if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged) return FR_E_INVAL;
  if (attr.device != plan->device) return FR_E_DEVICE_MISMATCH;
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  e = hipMemGetAddressRange(&base, &size, hipDeviceptr_t(const_cast<void*>(p)));
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return FR_E_INVAL;
  }
  const uintptr_t b = reinterpret_cast<uintptr_t>(base), q = reinterpret_cast<uintptr_t>(p);
  if (q < b || bytes > size || q - b > size - bytes) return FR_E_RANGE;
  return FR_OK;
}

bool overlap(const Region& x, const Region& y) {
  if (!x.p || !y.p || x.bytes == 0 || y.bytes == 0) return false;
  const uintptr_t a = reinterpret_cast<uintptr_t>(x.p), b = reinterpret_cast<uintptr_t>(y.p);
  return a < b + y.bytes && b < a + x.bytes;
}

// Outputs must not overlap each other or any input.
int check_disjoint(const Region* outs, int n_out, const Region* ins, int n_in) {
  for (int i = 0; i < n_out; i++) {
    for (int j = i + 1; j < n_out; j++)
      if (overlap(outs[i], outs[j])) return FR_E_OVERLAP;
    for (int j = 0; j < n_in; j++)
      if (overlap(outs[i], ins[j])) return FR_E_OVERLAP;
  }
  return FR_OK;
}

int launch_result(int hip_rc) {
  if (hip_rc == 0) return FR_OK;
  return device_error(hipError_t(hip_rc));
}

// The plan's pack / checksum / compare walk at the slice size of `tile`,
// line-aligned or not, in chunk order or (arena) in arena address order
// (the plan builds one for each configuration its operations use, so this
// finds one for the plan's own).
const SlotTable* src_walk(const fr_plan* plan, int tile, int line, int absorb, bool arena) {
  const uint32_t sl = slice_bytes(plan->layout.C, tile);
  const uint32_t shift = line_walk(plan, tile, line);
  const uint32_t ab = shift && absorb ? 1u : 0u;
  const bool order = arena && !plan->chunks_in_arena_order;
  for (const auto& w : plan->src_walks)
    if (w.sl == sl && w.t.shift == shift && w.t.absorb == ab && w.arena_order == order) return &w.t;
  return nullptr;
}

#define FR_TRY(expr)            \
  do {                          \
    const int rc_ = (expr);     \
    if (rc_ != FR_OK) return rc_; \
  } while (0)

}  // namespace

extern "C" int fr_pack_state(const fr_plan* plan, const void* src_base, void* payload,
                             uint64_t payload_cap, fr_chunk_sum* sums, hipStream_t stream) {
  if (!plan) return FR_E_INVAL;
  const Layout& L = plan->layout;
  if (payload_cap < L.payload_bytes) return FR_E_RANGE;
  FR_TRY(check_device_and_stream(plan, stream));
  FR_TRY(check_buffer(plan, src_base, plan->src_arena_bytes, 16));
  FR_TRY(check_buffer(plan, payload, L.payload_bytes, 16));
  FR_TRY(check_buffer(plan, sums, L.n_chunks * sizeof(fr_chunk_sum), 16));
  const Region outs[] = {{payload, L.payload_bytes}, {sums, L.n_chunks * sizeof(fr_chunk_sum)}};
  const Region ins[] = {{src_base, plan->src_arena_bytes}};
  FR_TRY(check_disjoint(outs, 2, ins, 1));
  if (plan->cfg.line_pack == kLineBlocks)
    return launch_result(launch_pack_blocks(plan->d_units, plan->pack_blocks, uint32_t(L.n_chunks),
                                            L.C, src_base, payload, sums, plan->scratch, plan->cfg,
                                            stream));
  const SlotTable* walk =
      src_walk(plan, plan->cfg.tile_pack, plan->cfg.line_pack, plan->cfg.absorb_pack, false);
  if (!walk) return FR_E_INVAL;
  return launch_result(launch_pack(plan->d_units, *walk, uint32_t(L.n_chunks), L.C, src_base,
                                   payload, sums, plan->scratch, plan->cfg, stream));
}

extern "C" int fr_unpack_state(const fr_plan* plan, const void* payload, const fr_chunk_sum* sums,
                               void* dst_base, uint32_t* bad_bitmap, uint64_t* n_bad,
                               hipStream_t stream) {
  if (!plan || !n_bad) return FR_E_INVAL;
  const Layout& L = plan->layout;
  const uint64_t words = (L.n_chunks + 31) / 32;
  FR_TRY(check_device_and_stream(plan, stream));
  FR_TRY(check_buffer(plan, payload, L.payload_bytes, 16));
  FR_TRY(check_buffer(plan, sums, L.n_chunks * sizeof(fr_chunk_sum), 16));
  FR_TRY(check_buffer(plan, dst_base, plan->dst_arena_bytes, 16));
  FR_TRY(check_buffer(plan, bad_bitmap, words * 4, 4));
  FR_TRY(check_buffer(plan, n_bad, 8, 8));
  const Region outs[] = {{dst_base, plan->dst_arena_bytes}, {bad_bitmap, words * 4}, {n_bad, 8}};
  const Region ins[] = {{payload, L.payload_bytes}, {sums, L.n_chunks * sizeof(fr_chunk_sum)}};
  FR_TRY(check_disjoint(outs, 3, ins, 2));
  UnpackArgs u;
  u.derived = plan->d_derived;
  u.n_derived = plan->n_derived;
  u.plain = plan->d_plain;
  u.n_plain = plan->n_plain;
  u.slots = plan->unpack_walk.t;
  u.n_chunks = uint32_t(L.n_chunks);
  u.C = L.C;
  u.payload = payload;
  u.sums = sums;
  u.dst = dst_base;
  u.bitmap = bad_bitmap;
  u.n_bad = n_bad;
  u.scratch = plan->scratch;
  if (plan->cfg.line_unpack == kLineBlocks)
    return launch_result(launch_unpack_blocks(u, plan->unpack_blocks, plan->cfg, stream));
  return launch_result(launch_unpack(u, plan->cfg, stream));
}

namespace {

// Argument checks of the replica compare (both entry points); on success
// *walk is the plan's compare walk.
int verify_checks(const fr_plan* plan, const void* base_a, const void* base_b,
                  uint32_t* diff_bitmap, uint64_t* n_diff, fr_chunk_sum* sums_a,
                  fr_chunk_sum* sums_b, hipStream_t stream, const SlotTable** walk) {
  if (!plan || !n_diff) return FR_E_INVAL;
  if ((sums_a == nullptr) != (sums_b == nullptr)) return FR_E_INVAL;
  const Layout& L = plan->layout;
  const uint64_t words = (L.n_chunks + 31) / 32;
  const uint64_t sb = sums_a ? L.n_chunks * sizeof(fr_chunk_sum) : 0;
  FR_TRY(check_device_and_stream(plan, stream));
  FR_TRY(check_buffer(plan, base_a, plan->src_arena_bytes, 16));
  FR_TRY(check_buffer(plan, base_b, plan->src_arena_bytes, 16));
  FR_TRY(check_buffer(plan, diff_bitmap, words * 4, 4));
  FR_TRY(check_buffer(plan, n_diff, 8, 8));
  if (sums_a) {
    FR_TRY(check_buffer(plan, sums_a, sb, 16));
    FR_TRY(check_buffer(plan, sums_b, sb, 16));
  }
  const Region outs[] = {{diff_bitmap, words * 4}, {n_diff, 8}, {sums_a, sb}, {sums_b, sb}};
  const Region ins[] = {{base_a, plan->src_arena_bytes}, {base_b, plan->src_arena_bytes}};
  FR_TRY(check_disjoint(outs, 4, ins, 2));
  *walk = src_walk(plan, plan->cfg.tile_verify, plan->cfg.line_verify, plan->cfg.absorb_verify,
                   plan->cfg.order_verify != 0);
  return *walk ? FR_OK : FR_E_INVAL;
}

}  // namespace

extern "C" int fr_verify_replicas(const fr_plan* plan, const void* base_a, const void* base_b,
                                  uint32_t* diff_bitmap, uint64_t* n_diff, fr_chunk_sum* sums_a,
                                  fr_chunk_sum* sums_b, hipStream_t stream) {
  const SlotTable* walk = nullptr;
  FR_TRY(verify_checks(plan, base_a, base_b, diff_bitmap, n_diff, sums_a, sums_b, stream, &walk));
  const Layout& L = plan->layout;
  return launch_result(launch_verify(plan->d_units, *walk, uint32_t(L.n_chunks), L.C, base_a,
                                     base_b, diff_bitmap, n_diff, sums_a, sums_b, plan->scratch,
                                     plan->cfg, stream));
}

extern "C" int fr_compare_sums(const fr_plan* plan, const fr_chunk_sum* sums_a,
                               const fr_chunk_sum* sums_b, uint32_t* diff_bitmap,
                               uint64_t* n_diff, hipStream_t stream) {
  if (!plan || !n_diff) return FR_E_INVAL;
  const Layout& L = plan->layout;
  const uint64_t words = (L.n_chunks + 31) / 32;
  const uint64_t sb = L.n_chunks * sizeof(fr_chunk_sum);
  FR_TRY(check_device_and_stream(plan, stream));
  FR_TRY(check_buffer(plan, sums_a, sb, 16));
  FR_TRY(check_buffer(plan, sums_b, sb, 16));
  FR_TRY(check_buffer(plan, diff_bitmap, words * 4, 4));
  FR_TRY(check_buffer(plan, n_diff, 8, 8));
  const Region outs[] = {{diff_bitmap, words * 4}, {n_diff, 8}};
  const Region ins[] = {{sums_a, sb}, {sums_b, sb}};
  FR_TRY(check_disjoint(outs, 2, ins, 2));
  return launch_result(
      launch_compare_sums(sums_a, sums_b, uint32_t(L.n_chunks), diff_bitmap, n_diff, stream));
}

extern "C" int fr_verify_replicas_noalloc(const fr_plan* plan, const void* base_a,
                                          const void* base_b, uint32_t* diff_bitmap,
                                          uint64_t* n_diff, fr_chunk_sum* sums_a,
                                          fr_chunk_sum* sums_b, hipStream_t stream) {
  const SlotTable* walk = nullptr;
  FR_TRY(verify_checks(plan, base_a, base_b, diff_bitmap, n_diff, sums_a, sums_b, stream, &walk));
  const Layout& L = plan->layout;
  // the same carving of the scratch as the plan's: flags, then the two
  // accumulator sets (only with sums)
  const uint64_t flag_bytes = (L.n_chunks * 4 + 255) & ~uint64_t(255);
  const uint64_t acc_bytes =
      sums_a ? L.n_chunks * accumulators_per_chunk(L.C, plan->cfg.tile_verify) * sizeof(fr_chunk_sum) : 0;
  if (flag_bytes > kStaticScratchBytes || 2 * acc_bytes > kStaticScratchBytes - flag_bytes)
    return FR_E_RANGE;
  void* base = nullptr;
  const int e = static_scratch_address(plan->device, &base);  // the plan's device is current
  if (e != 0) return device_error(hipError_t(e));
  uint8_t* p = static_cast<uint8_t*>(base);
  Scratch scr;
  scr.flags = reinterpret_cast<uint32_t*>(p);
  scr.acc = reinterpret_cast<fr_chunk_sum*>(p + flag_bytes);
  scr.acc_b = reinterpret_cast<fr_chunk_sum*>(p + flag_bytes + acc_bytes);
  return launch_result(launch_verify(plan->d_units, *walk, uint32_t(L.n_chunks), L.C, base_a,
                                     base_b, diff_bitmap, n_diff, sums_a, sums_b, scr, plan->cfg,
                                     stream));
}

extern "C" int fr_checksum_state(const fr_plan* plan, const void* base, fr_chunk_sum* sums,
                                 hipStream_t stream) {
  if (!plan) return FR_E_INVAL;
  const Layout& L = plan->layout;
  FR_TRY(check_device_and_stream(plan, stream));
  FR_TRY(check_buffer(plan, base, plan->src_arena_bytes, 16));
  FR_TRY(check_buffer(plan, sums, L.n_chunks * sizeof(fr_chunk_sum), 16));
  const Region outs[] = {{sums, L.n_chunks * sizeof(fr_chunk_sum)}};
  const Region ins[] = {{base, plan->src_arena_bytes}};
  FR_TRY(check_disjoint(outs, 1, ins, 1));
  const SlotTable* walk =
      src_walk(plan, plan->cfg.tile_checksum, plan->cfg.line_checksum, plan->cfg.absorb_checksum,
               plan->cfg.order_checksum != 0);
  if (!walk) return FR_E_INVAL;
  return launch_result(launch_checksum(plan->d_units, *walk, uint32_t(L.n_chunks), L.C, base,
                                       sums, plan->scratch, plan->cfg, stream));
}

// ------------------------------------------------------------ delta repair

namespace {

int check_list(const fr_plan* plan, const uint32_t* ids, uint64_t n_ids) {
  if (n_ids == 0) return FR_OK;
  if (!ids || n_ids > plan->layout.n_chunks) return FR_E_INVAL;
  for (uint64_t i = 0; i < n_ids; i++) {
    if (ids[i] >= plan->layout.n_chunks) return FR_E_INVAL;
    if (i && ids[i] <= ids[i - 1]) return FR_E_INVAL;
  }
  return FR_OK;
}

// Bytes of the delta payload of a host list: the listed chunks of sent
// entries in list order; a chunk right after the previous sent chunk of its
// entry follows it (that one is whole, so it ends on a multiple of C), any
// other starts at the next segment boundary; the end rounded up to 16.  Ids
// are strictly increasing (checked before), so one pass over the entries
// locates them all.
uint64_t delta_bytes(const fr_plan* plan, const uint32_t* ids, uint64_t n_ids) {
  const std::vector<uint64_t>& base = plan->layout.chunk_base;
  const uint64_t C = plan->layout.C, seg = plan->layout.seg;
  uint64_t end = 0, prev = ~uint64_t(0);  // the previous sent chunk's id
  uint32_t k = 0;
  for (uint64_t i = 0; i < n_ids; i++) {
    while (base[k + 1] <= ids[i]) k++;  // the entry with base[k] <= id < base[k + 1]
    const fr_tensor_desc& d = plan->table[k];
    if (d.derive_from >= 0) continue;
    const uint64_t j = ids[i] - base[k];
    const uint64_t nb = d.numel * (d.dtype == FR_F32 ? 4 : 2);
    const bool follows = j > 0 && prev == ids[i] - 1;
    const uint64_t at = follows ? end : (end + seg - 1) & ~(seg - 1);
    end = at + std::min<uint64_t>(C, nb - j * C);
    prev = ids[i];
  }
  return (end + 15) & ~uint64_t(15);
}

// Implicit walk over a list of at most `bound` units whose length the device
// holds at *count (derived groups: two chunks' worth of master slices each),
// at the slice size of `tile`.
SlotTable list_walk(uint64_t bound, const uint64_t* count, uint64_t C, int tile, bool derived) {
  uint32_t sh = 0;
  while ((uint64_t(slice_bytes(C, tile)) << sh) < C) sh++;
  SlotTable t;
  t.implicit_shift = sh + (derived ? 1 : 0);
  t.n = bound << t.implicit_shift;
  t.count = count;
  return t;
}

// Enqueues the upload of a host list into the plan's device list and its
// bitmap.  The list goes through the plan's pinned staging; the staging is
// refilled only after the previous upload from it has completed (an event
// recorded behind each copy).
int upload_list(const fr_plan* plan, const uint32_t* ids, uint64_t n_ids, hipStream_t stream) {
  hipError_t e = hipEventSynchronize(plan->delta_ids_copied);
  if (e != hipSuccess) return device_error(e);
  std::memcpy(plan->h_delta_ids, ids, n_ids * sizeof(uint32_t));
  e = hipMemcpyAsync(plan->d_delta_ids, plan->h_delta_ids, n_ids * sizeof(uint32_t),
                     hipMemcpyHostToDevice, stream);
  if (e == hipSuccess) e = hipEventRecord(plan->delta_ids_copied, stream);
  if (e != hipSuccess) return device_error(e);
  const uint64_t words = (plan->layout.n_chunks + 31) / 32;
  return launch_result(launch_ids_to_bits(plan->d_delta_ids, n_ids, plan->d_delta_bits, words, stream));
}

// Arguments of the list builder for a call of operation `tile` (whose
// accumulators per list position it clears, with *zero_word if given).
DeltaBuild delta_build(const fr_plan* plan, const uint32_t* bits, uint64_t* user_counts,
                       uint64_t payload_limit, int tile, uint64_t* zero_word) {
  DeltaBuild b{};
  b.loc = plan->d_delta_loc;
  b.bits = bits;
  b.n_chunks = plan->layout.n_chunks;
  b.seg = plan->layout.seg;
  b.agg = plan->d_delta_agg;
  b.pre = plan->d_delta_pre;
  b.counts = plan->d_delta_counts;
  b.user_counts = user_counts;
  b.src_units = plan->d_delta_src;
  b.plain = plan->d_delta_plain;
  b.derived = plan->d_delta_derived;
  b.bad = plan->scratch.flags;
  b.pay_of = plan->d_delta_payof;
  b.m0 = plan->d_delta_m0;
  b.payload_limit = payload_limit;
  b.acc = plan->scratch.acc;
  uint32_t g = 0;
  while ((uint64_t(1) << g) < accumulators_per_chunk(plan->layout.C, tile)) g++;
  b.acc_shift = g;
  b.zero_word = zero_word;
  return b;
}

// The device half of a delta pack: build the list's records from `bits`,
// then pack them (at most `bound` units).
int pack_list(const fr_plan* plan, const void* src_base, const uint32_t* bits, uint64_t bound,
              void* payload, uint64_t payload_cap, fr_chunk_sum* sums, uint64_t* user_counts,
              hipStream_t stream) {
  FR_TRY(launch_result(launch_delta_build(
      delta_build(plan, bits, user_counts, payload_cap, plan->cfg.tile_pack, nullptr), true, stream)));
  const uint64_t C = plan->layout.C;
  return launch_result(launch_pack(plan->d_delta_src,
                                   list_walk(bound, plan->d_delta_counts + kDeltaIds, C,
                                             plan->cfg.tile_pack, false),
                                   uint32_t(bound), C, src_base, payload, sums, plan->scratch,
                                   plan->cfg, stream));
}

// The device half of a delta unpack: build the list's records from `bits`,
// write the sent chunks and re-derive the listed parameters (from re-sent
// masters in the payload, else from the receiver's own) in one launch,
// check every listed chunk (at most `bound`).
int unpack_list(const fr_plan* plan, const void* payload, uint64_t payload_bytes,
                const fr_chunk_sum* sums, const uint32_t* bits, uint64_t bound, void* dst_base,
                uint32_t* bad_bitmap, uint64_t* n_bad, hipStream_t stream) {
  if (bound) {
    FR_TRY(launch_result(launch_delta_build(
        delta_build(plan, bits, nullptr, payload_bytes, plan->cfg.tile_unpack, n_bad), false, stream)));
  }
  const uint64_t C = plan->layout.C;
  UnpackDeltaArgs a{};
  a.plain = plan->d_delta_plain;
  a.n_plain = 0;
  a.derived = plan->d_delta_derived;
  a.n_derived = 0;
  a.plain_slots = list_walk(bound, plan->d_delta_counts + kDeltaSent, C, plan->cfg.tile_unpack, false);
  a.derived_slots = list_walk(bound, plan->d_delta_counts + kDeltaDerived, C, plan->cfg.tile_unpack, true);
  a.n_ids = uint32_t(bound);
  a.C = C;
  a.payload = payload;
  a.sums = sums;
  a.dst = dst_base;
  a.bitmap = bad_bitmap;
  a.n_bad = n_bad;
  a.scratch = plan->scratch;
  if (bound) {  // the builder cleared the accumulators and n_bad
    a.live = plan->d_delta_counts + kDeltaIds;
    a.bad = plan->scratch.flags;
  }
  a.bits = bits;
  a.pay_of = plan->d_delta_payof;
  return launch_result(launch_unpack_delta(a, plan->cfg, stream));
}

}  // namespace

extern "C" int fr_delta_layout(const fr_plan* plan, const uint32_t* ids, uint64_t n_ids,
                               uint64_t* payload_bytes) {
  if (!plan || !payload_bytes) return FR_E_INVAL;
  FR_TRY(check_list(plan, ids, n_ids));
  *payload_bytes = delta_bytes(plan, ids, n_ids);
  return FR_OK;
}

extern "C" int fr_pack_chunks(const fr_plan* plan, const void* src_base, const uint32_t* ids,
                              uint64_t n_ids, void* payload, uint64_t payload_cap,
                              fr_chunk_sum* sums, hipStream_t stream) {
  if (!plan) return FR_E_INVAL;
  FR_TRY(check_list(plan, ids, n_ids));
  const uint64_t pb = delta_bytes(plan, ids, n_ids);
  if (payload_cap < pb) return FR_E_RANGE;
  FR_TRY(check_device_and_stream(plan, stream));
  FR_TRY(check_buffer(plan, src_base, plan->src_arena_bytes, 16));
  FR_TRY(check_buffer(plan, payload, pb, 16));
  FR_TRY(check_buffer(plan, sums, n_ids * sizeof(fr_chunk_sum), 16));
  const Region outs[] = {{payload, pb}, {sums, n_ids * sizeof(fr_chunk_sum)}};
  const Region ins[] = {{src_base, plan->src_arena_bytes}};
  FR_TRY(check_disjoint(outs, 2, ins, 1));
  if (n_ids == 0) return FR_OK;
  FR_TRY(upload_list(plan, ids, n_ids, stream));
  return pack_list(plan, src_base, plan->d_delta_bits, n_ids, payload, pb, sums, nullptr, stream);
}

extern "C" int fr_unpack_chunks(const fr_plan* plan, const void* payload, uint64_t payload_bytes,
                                const fr_chunk_sum* sums, const uint32_t* ids, uint64_t n_ids,
                                void* dst_base, uint32_t* bad_bitmap, uint64_t* n_bad,
                                hipStream_t stream) {
  if (!plan || !n_bad) return FR_E_INVAL;
  FR_TRY(check_list(plan, ids, n_ids));
  const uint64_t pb = delta_bytes(plan, ids, n_ids);
  if (payload_bytes < pb) return FR_E_RANGE;
  const uint64_t words = (n_ids + 31) / 32;
  FR_TRY(check_device_and_stream(plan, stream));
  FR_TRY(check_buffer(plan, payload, pb, 16));
  FR_TRY(check_buffer(plan, sums, n_ids * sizeof(fr_chunk_sum), 16));
  FR_TRY(check_buffer(plan, dst_base, plan->dst_arena_bytes, 16));
  FR_TRY(check_buffer(plan, bad_bitmap, words * 4, 4));
  FR_TRY(check_buffer(plan, n_bad, 8, 8));
  const Region outs[] = {{dst_base, plan->dst_arena_bytes}, {bad_bitmap, words * 4}, {n_bad, 8}};
  const Region ins[] = {{payload, pb}, {sums, n_ids * sizeof(fr_chunk_sum)}};
  FR_TRY(check_disjoint(outs, 3, ins, 2));
  if (n_ids) FR_TRY(upload_list(plan, ids, n_ids, stream));
  return unpack_list(plan, payload, pb, sums, plan->d_delta_bits, n_ids, dst_base, bad_bitmap,
                     n_bad, stream);
}

extern "C" int fr_pack_flagged(const fr_plan* plan, const void* src_base, const uint32_t* flagged,
                               void* payload, uint64_t payload_cap, fr_chunk_sum* sums,
                               uint64_t* counts, hipStream_t stream) {
  if (!plan) return FR_E_INVAL;
  const Layout& L = plan->layout;
  const uint64_t words = (L.n_chunks + 31) / 32, pmax = L.delta_payload_max;
  if (payload_cap < pmax) return FR_E_RANGE;
  FR_TRY(check_device_and_stream(plan, stream));
  FR_TRY(check_buffer(plan, src_base, plan->src_arena_bytes, 16));
  FR_TRY(check_buffer(plan, flagged, words * 4, 4));
  FR_TRY(check_buffer(plan, payload, pmax, 16));
  FR_TRY(check_buffer(plan, sums, L.n_chunks * sizeof(fr_chunk_sum), 16));
  if (counts) FR_TRY(check_buffer(plan, counts, 16, 8));
  const Region outs[] = {{payload, pmax}, {sums, L.n_chunks * sizeof(fr_chunk_sum)}, {counts, counts ? 16u : 0u}};
  const Region ins[] = {{src_base, plan->src_arena_bytes}, {flagged, words * 4}};
  FR_TRY(check_disjoint(outs, 3, ins, 2));
  return pack_list(plan, src_base, flagged, L.n_chunks, payload, pmax, sums, counts, stream);
}

extern "C" int fr_unpack_flagged(const fr_plan* plan, const void* payload, uint64_t payload_bytes,
                                 const fr_chunk_sum* sums, const uint32_t* flagged, void* dst_base,
                                 uint32_t* bad_bitmap, uint64_t* n_bad, hipStream_t stream) {
  if (!plan || !n_bad) return FR_E_INVAL;
  const Layout& L = plan->layout;
  const uint64_t words = (L.n_chunks + 31) / 32;
  FR_TRY(check_device_and_stream(plan, stream));
  if (payload_bytes) FR_TRY(check_buffer(plan, payload, payload_bytes, 16));
  FR_TRY(check_buffer(plan, sums, L.n_chunks * sizeof(fr_chunk_sum), 16));
  FR_TRY(check_buffer(plan, flagged, words * 4, 4));
  FR_TRY(check_buffer(plan, dst_base, plan->dst_arena_bytes, 16));
  FR_TRY(check_buffer(plan, bad_bitmap, words * 4, 4));
  FR_TRY(check_buffer(plan, n_bad, 8, 8));
  const Region outs[] = {{dst_base, plan->dst_arena_bytes}, {bad_bitmap, words * 4}, {n_bad, 8}};
  const Region ins[] = {{payload, payload_bytes}, {sums, L.n_chunks * sizeof(fr_chunk_sum)},
                        {flagged, words * 4}};
  FR_TRY(check_disjoint(outs, 3, ins, 3));
  return unpack_list(plan, payload, payload_bytes, sums, flagged, L.n_chunks, dst_base, bad_bitmap,
                     n_bad, stream);
}

extern "C" const char* fr_strerror(int status) {
  switch (status) {
    case FR_OK: return "ok";
    case FR_E_INVAL: return "invalid argument";
    case FR_E_ALIGN: return "misaligned offset or pointer";
    case FR_E_RANGE: return "out of range";
    case FR_E_OVERLAP: return "overlapping ranges or buffers";
    case FR_E_NOMEM: return "out of memory";
    case FR_E_DEVICE: return "HIP error";
    case FR_E_DEVICE_MISMATCH: return "device mismatch";
    default: return "unknown status";
  }
}

extern "C" int fr_last_hip_error(void) { return g_last_hip_error; }

extern "C" int fr_abi_version(void) { return FR_ABI_VERSION; }
