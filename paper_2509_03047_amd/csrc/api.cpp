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
// line-aligned or not (the plan builds one for each configuration its
// operations use, so this finds one for the plan's own).
const SlotTable* src_walk(const fr_plan* plan, int tile, int line) {
  const uint32_t sl = slice_bytes(plan->layout.C, tile);
  const uint32_t shift = line_walk(plan, tile, line);
  for (const auto& w : plan->src_walks)
    if (w.sl == sl && w.t.shift == shift) return &w.t;
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
  const SlotTable* walk = src_walk(plan, plan->cfg.tile_pack, plan->cfg.line_pack);
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
  *walk = src_walk(plan, plan->cfg.tile_verify, plan->cfg.line_verify);
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
  const SlotTable* walk = src_walk(plan, plan->cfg.tile_checksum, plan->cfg.line_checksum);
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

struct Where {
  uint32_t entry;
  uint64_t j;    // chunk index within the entry
  uint64_t len;  // chunk bytes
};

// Delta payload layout: the listed chunks of sent entries in list order; a
// chunk right after the previous sent chunk of its entry follows it (that
// one is whole, so it ends on a multiple of C), any other starts at the next
// segment boundary; the payload ends at the last chunk's end rounded up to
// 16.  Ids are strictly increasing (checked before), so one pass over the
// entries locates them all.
struct DeltaList {
  std::vector<Where> where;   // per list position
  std::vector<uint64_t> off;  // payload offset per list position (kNoPayload: derived)
  uint64_t bytes = 0;         // payload bytes
};

void delta_layout(const fr_plan* plan, const uint32_t* ids, uint64_t n_ids, DeltaList* out) {
  const std::vector<uint64_t>& base = plan->layout.chunk_base;
  const uint64_t C = plan->layout.C;
  out->where.resize(n_ids);
  out->off.assign(n_ids, kNoPayload);
  uint64_t end = 0;
  bool have_prev = false;
  Where prev{};
  uint32_t k = 0;
  for (uint64_t i = 0; i < n_ids; i++) {
    while (base[k + 1] <= ids[i]) k++;  // the entry with base[k] <= id < base[k + 1]
    const fr_tensor_desc& d = plan->table[k];
    const uint64_t nb = d.numel * (d.dtype == FR_F32 ? 4 : 2);
    const uint64_t j = ids[i] - base[k];
    const Where w{k, j, std::min<uint64_t>(C, nb - j * C)};
    out->where[i] = w;
    if (d.derive_from >= 0) continue;
    const bool follows = have_prev && prev.entry == w.entry && prev.j + 1 == w.j;
    const uint64_t seg = plan->layout.seg;
    const uint64_t at = follows ? end : (end + seg - 1) & ~(seg - 1);
    out->off[i] = at;
    end = at + w.len;
    prev = w;
    have_prev = true;
  }
  out->bytes = (end + 15) & ~uint64_t(15);
}

// Device buffer for a delta call's records and slot tables.  It grows on
// demand; before the old one is freed, the device is synchronised, since
// work enqueued by earlier calls (on any stream) may still read it.
int ensure_delta_buffer(fr_plan* plan, uint64_t need) {
  if (plan->d_delta && plan->delta_cap >= need) return FR_OK;
  if (plan->d_delta) {
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return device_error(e);
    (void)hipFree(plan->d_delta);
    plan->d_delta = nullptr;
    plan->delta_cap = 0;
  }
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, need);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e == hipErrorOutOfMemory ? FR_E_NOMEM : device_error(e);
  }
  plan->d_delta = p;
  plan->delta_cap = need;
  return FR_OK;
}

// Implicit walk over `units` chunks (derived groups: two chunks' worth of
// master slices each) at the slice size of `tile`.
SlotTable implicit_walk(uint64_t units, uint64_t C, int tile, bool derived) {
  uint32_t sh = 0;
  while ((uint64_t(slice_bytes(C, tile)) << sh) < C) sh++;
  SlotTable t;
  t.implicit_shift = sh + (derived ? 1 : 0);
  t.n = units << t.implicit_shift;
  return t;
}

// The staging vector is pageable memory, and HIP performs an async copy from
// pageable memory synchronously: the records have left the vector when this
// returns, so the next delta call may refill or reallocate it at once.
int upload_records(fr_plan* plan, size_t bytes, hipStream_t stream) {
  if (bytes == 0) return FR_OK;
  hipError_t e = hipMemcpyAsync(plan->d_delta, plan->delta_host.data(), bytes,
                                hipMemcpyHostToDevice, hipStream_t(stream));
  return e == hipSuccess ? FR_OK : device_error(e);
}

}  // namespace

extern "C" int fr_delta_layout(const fr_plan* plan, const uint32_t* ids, uint64_t n_ids,
                               uint64_t* payload_bytes) {
  if (!plan || !payload_bytes) return FR_E_INVAL;
  FR_TRY(check_list(plan, ids, n_ids));
  DeltaList dl;
  try {
    delta_layout(plan, ids, n_ids, &dl);
  } catch (const std::bad_alloc&) {
    return FR_E_NOMEM;
  }
  *payload_bytes = dl.bytes;
  return FR_OK;
}

extern "C" int fr_pack_chunks(const fr_plan* cplan, const void* src_base, const uint32_t* ids,
                              uint64_t n_ids, void* payload, uint64_t payload_cap,
                              fr_chunk_sum* sums, hipStream_t stream) {
  if (!cplan) return FR_E_INVAL;
  fr_plan* plan = const_cast<fr_plan*>(cplan);  // the plan's delta staging is mutable state
  FR_TRY(check_list(plan, ids, n_ids));
  DeltaList dl;
  try {
    delta_layout(plan, ids, n_ids, &dl);
  } catch (const std::bad_alloc&) {
    return FR_E_NOMEM;
  }
  const uint64_t pb = dl.bytes;
  if (payload_cap < pb) return FR_E_RANGE;
  FR_TRY(check_device_and_stream(plan, stream));
  FR_TRY(check_buffer(plan, src_base, plan->src_arena_bytes, 16));
  FR_TRY(check_buffer(plan, payload, pb, 16));
  FR_TRY(check_buffer(plan, sums, n_ids * sizeof(fr_chunk_sum), 16));
  const Region outs[] = {{payload, pb}, {sums, n_ids * sizeof(fr_chunk_sum)}};
  const Region ins[] = {{src_base, plan->src_arena_bytes}};
  FR_TRY(check_disjoint(outs, 2, ins, 1));
  if (n_ids == 0) return FR_OK;
  const uint64_t C = plan->layout.C;
  try {
    plan->delta_host.resize(n_ids * sizeof(SrcUnit));
  } catch (const std::bad_alloc&) {
    return FR_E_NOMEM;
  }
  SrcUnit* recs = reinterpret_cast<SrcUnit*>(plan->delta_host.data());
  for (uint64_t i = 0, last_sent = n_ids; i < n_ids; i++) {
    const Where& w = dl.where[i];
    SrcUnit& r = recs[i];
    r = SrcUnit{};
    r.src_off = plan->table[w.entry].src_offset + w.j * C;
    r.len = uint32_t(w.len);
    r.c = uint32_t(i);
    r.pay_off = dl.off[i];
    if (dl.off[i] == kNoPayload) continue;
    if (last_sent < n_ids) {  // the previous sent chunk zero-fills up to this one
      SrcUnit& p = recs[last_sent];
      p.gap_v = uint32_t((dl.off[i] - ((p.pay_off + p.len + 15) & ~uint64_t(15))) >> 4);
    }
    last_sent = i;
  }
  FR_TRY(ensure_delta_buffer(plan, plan->delta_host.size()));
  FR_TRY(upload_records(plan, plan->delta_host.size(), stream));
  return launch_result(launch_pack(static_cast<const SrcUnit*>(plan->d_delta),
                                   implicit_walk(n_ids, C, plan->cfg.tile_pack, false),
                                   uint32_t(n_ids), C, src_base, payload, sums, plan->scratch,
                                   plan->cfg, stream));
}

extern "C" int fr_unpack_chunks(const fr_plan* cplan, const void* payload,
                                uint64_t payload_bytes, const fr_chunk_sum* sums,
                                const uint32_t* ids, uint64_t n_ids, void* dst_base,
                                uint32_t* bad_bitmap, uint64_t* n_bad, hipStream_t stream) {
  if (!cplan || !n_bad) return FR_E_INVAL;
  fr_plan* plan = const_cast<fr_plan*>(cplan);
  FR_TRY(check_list(plan, ids, n_ids));
  DeltaList dl;
  try {
    delta_layout(plan, ids, n_ids, &dl);
  } catch (const std::bad_alloc&) {
    return FR_E_NOMEM;
  }
  const uint64_t pb = dl.bytes;
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
  const uint64_t C = plan->layout.C;
  uint32_t n_plain = 0, n_derived = 0;
  for (uint64_t i = 0; i < n_ids; i++) (dl.off[i] == kNoPayload ? n_derived : n_plain)++;
  try {
    plan->delta_host.resize(n_plain * sizeof(PlainUnit) + n_derived * sizeof(DerivedUnit));
  } catch (const std::bad_alloc&) {
    return FR_E_NOMEM;
  }
  // device image: [plain units][derived units]
  PlainUnit* pu = reinterpret_cast<PlainUnit*>(plan->delta_host.data());
  DerivedUnit* du = reinterpret_cast<DerivedUnit*>(plan->delta_host.data() + n_plain * sizeof(PlainUnit));
  uint32_t ip = 0, id = 0;
  for (uint64_t i = 0; i < n_ids; i++) {
    const Where& w = dl.where[i];
    const fr_tensor_desc& d = plan->table[w.entry];
    if (d.derive_from < 0) {
      PlainUnit& u = pu[ip++];
      u = PlainUnit{};
      u.pay_off = dl.off[i];
      u.dst_off = d.dst_offset + w.j * C;
      u.len = uint32_t(w.len);
      u.c = uint32_t(i);
    } else {
      const fr_tensor_desc& m = plan->table[d.derive_from];
      DerivedUnit& u = du[id++];
      u = DerivedUnit{};
      u.m_pay_off = m.dst_offset + 2 * w.j * C;  // the receiver's master bytes of this chunk
      u.m_dst_off = u.m_pay_off;
      u.p_dst_off = d.dst_offset + w.j * C;
      u.len = uint32_t(w.len);
      u.c = uint32_t(i);
    }
  }
  if (n_ids) {
    FR_TRY(ensure_delta_buffer(plan, plan->delta_host.size()));
    FR_TRY(upload_records(plan, plan->delta_host.size(), stream));
  }
  UnpackDeltaArgs a{};
  a.plain = static_cast<const PlainUnit*>(plan->d_delta);
  a.n_plain = n_plain;
  a.derived = reinterpret_cast<const DerivedUnit*>(static_cast<const uint8_t*>(plan->d_delta) +
                                                   n_plain * sizeof(PlainUnit));
  a.n_derived = n_derived;
  a.plain_slots = implicit_walk(n_plain, C, plan->cfg.tile_unpack, false);
  a.derived_slots = implicit_walk(n_derived, C, plan->cfg.tile_unpack, true);
  a.n_ids = uint32_t(n_ids);
  a.C = C;
  a.payload = payload;
  a.sums = sums;
  a.dst = dst_base;
  a.bitmap = bad_bitmap;
  a.n_bad = n_bad;
  a.scratch = plan->scratch;
  return launch_result(launch_unpack_delta(a, plan->cfg, stream));
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
