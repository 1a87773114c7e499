// Plan: validation of a tensor table, the chunk / payload layout, and the
// device tables the kernels walk: unit records (one SrcUnit per chunk for
// pack, checksum and replica compare; derived groups and plain chunks for
// unpack) and the slot tables that walk them.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <new>
#include <utility>
#include <vector>

#include "fr_internal.h"

namespace fr {

thread_local int g_last_hip_error = 0;

// Default tile of each operation (kernels.hip: 4 = 64 threads x 4 vectors,
// 5 = 128 threads x 2 vectors, both 4 KiB slices; 3 = 256 threads x 4
// vectors, 16 KiB slices), chosen by sweeping all tiles on MI355X over the
// 8B and 70B rank shares and the descriptor stress table.
constexpr uint32_t kDefaultTilePack = 4, kDefaultTileUnpack = 5, kDefaultTileVerify = 5,
                   kDefaultTileChecksum = 3;

// The tile an operation takes for chunks of C bytes when no tile variable is
// set: the default above, except that chunks smaller than its slice would
// leave most lanes idle, so smaller chunks take smaller tiles (sweeps of
// seven tiles at 1-8 KiB chunks on the 8B share and the stress table:
// unpack 2.7 -> 4.1 TB/s at 1 KiB with 64 x 1, compare 3.8 -> 7.2, the
// checksum 1.0 -> 3.2 at 1 KiB and 3.8 -> 6.6 at 4 KiB with 64 x 4; pack is
// as fast with its default at every size).
enum TileOp { kOpPack, kOpUnpack, kOpVerify, kOpChecksum };
int auto_tile(TileOp op, uint64_t C) {
  switch (op) {
    case kOpUnpack: return C <= 1024 ? 7 : C <= 2048 ? 6 : int(kDefaultTileUnpack);
    case kOpVerify: return C <= 2048 ? 7 : int(kDefaultTileVerify);
    case kOpChecksum: return C <= 4096 ? 4 : C <= 8192 ? 9 : int(kDefaultTileChecksum);
    default: return int(kDefaultTilePack);
  }
}
// Walks (0 plain; 1 cut at lines of the arena read, for unpack of the
// receiver; 2 at lines of the payload; 4 by blocks of the payload): pack and
// unpack by payload blocks when payload chunks start inside lines (16-byte
// segments of tensors whose sizes are not multiples of 128 bytes), else pack
// at payload lines and unpack at receiver lines (both plain walks when every
// chunk starts on a line); the compare at arena lines.
constexpr int kDefaultLinePack = kLineAuto, kDefaultLineUnpack = kLineAuto, kDefaultLineVerify = 1,
              kDefaultLineChecksum = 0;
constexpr int kAlignedLinePack = 2, kAlignedLineUnpack = 1;
// Slice walks loading through buffer resources (every load of a thread in
// flight at once) instead of predicated global loads: off by default.  On
// MI355X they made pack 2.5 % slower and the stress table's pack 2-3 %
// faster (the block walk that table takes is faster still), unpack 1.5-2.5 %
// slower, the checksum no faster, and the compare between 0.5 % slower and
// 1.3 % faster from one box to the next.
constexpr uint32_t kDefaultBufPack = 0, kDefaultBufUnpack = 0, kDefaultBufVerify = 0,
                   kDefaultBufChecksum = 0;
// The compare's and the checksum's walks in arena address order instead of
// chunk order, for tables that list tensors out of arena order: on the
// descriptor stress table the compare gains 2.8 % (7.19 against 6.99 TB/s)
// and the checksum loses 1.1 % (6.50 against 6.57).
constexpr uint32_t kDefaultOrderVerify = 1, kDefaultOrderChecksum = 0;
// Whether a line-aligned pack / unpack walk lets a unit's last slice absorb
// the lead instead of adding a slice.
constexpr uint32_t kDefaultAbsorbPack = 1, kDefaultAbsorbUnpack = 1, kDefaultAbsorbVerify = 0,
                   kDefaultAbsorbChecksum = 0;
// Workgroups of a launch that walks a delta list built on the device (the
// host knows only its largest possible length): 256 per CU.
constexpr uint32_t kDefaultDeltaGrid = 65536;

static uint64_t esize(uint32_t dtype) { return dtype == FR_F32 ? 4 : 2; }
static uint64_t align16(uint64_t x) { return (x + 15) & ~uint64_t(15); }
static uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) & ~(a - 1); }

int validate_and_layout(const fr_tensor_desc* t, uint32_t n, uint64_t C, uint64_t seg,
                        uint64_t src_bytes, uint64_t dst_bytes, Layout* L) {
  if (n > 0 && t == nullptr) return FR_E_INVAL;
  if (n > 0x7FFFFFFFu) return FR_E_INVAL;
  if (C < 16 || C > (uint64_t(1) << 30) || (C & (C - 1)) != 0) return FR_E_INVAL;
  if (seg < 16 || seg > kMaxSegmentAlign || (seg & (seg - 1)) != 0) return FR_E_INVAL;
  // Field checks, in an order that makes the reported error deterministic:
  // dtype and derive_from first (INVAL), then alignment, then ranges.
  std::vector<uint8_t> used_as_master(n, 0);
  for (uint32_t k = 0; k < n; k++) {
    const fr_tensor_desc& e = t[k];
    if (e.dtype != FR_F32 && e.dtype != FR_BF16) return FR_E_INVAL;
    if (e.numel > (uint64_t(1) << 61)) return FR_E_RANGE;
    if (e.derive_from != -1) {
      if (e.derive_from < 0 || uint32_t(e.derive_from) >= n || uint32_t(e.derive_from) == k)
        return FR_E_INVAL;
      const fr_tensor_desc& m = t[e.derive_from];
      if (e.dtype != FR_BF16 || m.dtype != FR_F32 || m.derive_from != -1 || m.numel != e.numel)
        return FR_E_INVAL;
      if (used_as_master[e.derive_from]) return FR_E_INVAL;
      used_as_master[e.derive_from] = 1;
    }
  }
  for (uint32_t k = 0; k < n; k++)
    if ((t[k].src_offset | t[k].dst_offset) & 15) return FR_E_ALIGN;
  uint64_t state = 0;
  for (uint32_t k = 0; k < n; k++) {
    uint64_t nb = t[k].numel * esize(t[k].dtype);
    if (t[k].src_offset > src_bytes || nb > src_bytes - t[k].src_offset) return FR_E_RANGE;
    if (t[k].dst_offset > dst_bytes || nb > dst_bytes - t[k].dst_offset) return FR_E_RANGE;
    state += nb;
  }
  // Receiver ranges must be disjoint: unpack writes every one of them.
  std::vector<std::pair<uint64_t, uint64_t>> ranges;
  ranges.reserve(n);
  for (uint32_t k = 0; k < n; k++) {
    uint64_t nb = t[k].numel * esize(t[k].dtype);
    if (nb) ranges.emplace_back(t[k].dst_offset, t[k].dst_offset + nb);
  }
  std::sort(ranges.begin(), ranges.end());
  for (size_t i = 1; i < ranges.size(); i++)
    if (ranges[i].first < ranges[i - 1].second) return FR_E_OVERLAP;

  L->C = C;
  L->seg = seg;
  L->pay_off.assign(n, 0);
  L->chunk_base.assign(size_t(n) + 1, 0);
  uint64_t base = 0, end = 0;  // end of the last payload segment so far
  uint64_t sent_bytes = 0;
  L->n_sent_chunks = 0;
  for (uint32_t k = 0; k < n; k++) {
    uint64_t nb = t[k].numel * esize(t[k].dtype);
    L->chunk_base[k] = base;
    base += (nb + C - 1) / C;
    if (t[k].derive_from < 0) {
      L->n_sent_chunks += (nb + C - 1) / C;
      sent_bytes += nb;
    }
    if (t[k].derive_from >= 0) {
      L->pay_off[k] = kNoPayload;
    } else if (nb == 0) {
      L->pay_off[k] = align16(end);  // an empty entry occupies no segment
    } else {
      L->pay_off[k] = align_up(end, seg);
      end = L->pay_off[k] + nb;
    }
  }
  L->chunk_base[n] = base;
  if (base > 0xFFFFFFFFull) return FR_E_RANGE;  // chunk ids are 32-bit
  L->n_chunks = base;
  L->payload_bytes = align16(end);
  L->state_bytes = state;
  // A delta payload never outgrows the full one when C >= A: chunk by chunk
  // its offsets stay at or below the full payload's, whose chunks all start
  // on multiples of A.  With C < A each sent chunk adds at most its bytes and
  // a gap below A.
  L->delta_payload_max = C >= seg ? L->payload_bytes : align16(sent_bytes + L->n_sent_chunks * seg);
  return FR_OK;
}

static void fill_info(const Layout& L, uint32_t n, uint64_t src, uint64_t dst, int64_t dev,
                      const LaunchCfg& cfg, fr_plan_info* info, uint32_t pack_walk = 0,
                      uint32_t unpack_walk = 0) {
  info->n_entries = n;
  info->chunk_bytes = L.C;
  info->n_chunks = L.n_chunks;
  info->payload_bytes = L.payload_bytes;
  info->bitmap_words = (L.n_chunks + 31) / 32;
  info->src_arena_bytes = src;
  info->dst_arena_bytes = dst;
  info->state_bytes = L.state_bytes;
  info->device = dev;
  info->segment_align = L.seg;
  info->delta_payload_max = L.delta_payload_max;
  info->pack_walk = pack_walk;
  info->unpack_walk = unpack_walk;
  info->tile_pack = uint32_t(cfg.tile_pack);
  info->tile_unpack = uint32_t(cfg.tile_unpack);
  info->tile_verify = uint32_t(cfg.tile_verify);
  info->tile_checksum = uint32_t(cfg.tile_checksum);
}

static uint32_t env_u32(const char* name, uint32_t dflt) {
  const char* v = std::getenv(name);
  if (!v || !*v) return dflt;
  char* end = nullptr;
  unsigned long x = std::strtoul(v, &end, 10);
  return (end && *end == 0) ? uint32_t(x) : dflt;
}

}  // namespace fr

using namespace fr;

static LaunchCfg plan_launch_config(uint64_t C);

extern "C" int fr_layout_query(const fr_tensor_desc* table, uint32_t n, uint64_t C,
                               uint64_t src_bytes, uint64_t dst_bytes, uint64_t seg,
                               fr_plan_info* info, uint64_t* payload_offset,
                               uint64_t* chunk_base) {
  if (!info) return FR_E_INVAL;
  Layout L;
  int rc;
  try {
    rc = validate_and_layout(table, n, C, seg, src_bytes, dst_bytes, &L);
  } catch (const std::bad_alloc&) {
    return FR_E_NOMEM;
  }
  if (rc != FR_OK) return rc;
  fill_info(L, n, src_bytes, dst_bytes, -1, plan_launch_config(C), info);
  if (payload_offset && n) std::memcpy(payload_offset, L.pay_off.data(), sizeof(uint64_t) * n);
  if (chunk_base) std::memcpy(chunk_base, L.chunk_base.data(), sizeof(uint64_t) * (size_t(n) + 1));
  return FR_OK;
}

static int hip_fail(hipError_t e) {
  g_last_hip_error = int(e);
  return FR_E_DEVICE;
}

// Plan creation works on a stream of its own that does not synchronise with
// the null stream, and frees nothing on success (hipFree waits for the whole
// device), so that creating a plan does not stall other work on the device.
// `runs` stages the run descriptions of the slot tables; it points into the
// plan's scratch, which no call has used yet and every call clears first.
struct Staging {
  hipStream_t s = nullptr;
  uint64_t* runs = nullptr;
  uint64_t runs_cap = 0;  // in uint64_t
  ~Staging() {
    if (s) (void)hipStreamDestroy(s);
  }
};

// Host-to-device copy on the creation stream, finished before returning (the
// host arrays are temporaries of the caller).
static int copy_in(void* dst, const void* src, size_t bytes, hipStream_t s) {
  if (bytes == 0) return FR_OK;
  hipError_t e = hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  return e == hipSuccess ? FR_OK : hip_fail(e);
}

// Device copy of a host array (or an uninitialised buffer when src is NULL).
static int upload(const void* src, size_t bytes, void** out, hipStream_t s) {
  *out = nullptr;
  if (bytes == 0) return FR_OK;
  hipError_t e = hipMalloc(out, bytes);
  if (e != hipSuccess) {
    *out = nullptr;
    (void)hipGetLastError();
    return e == hipErrorOutOfMemory ? FR_E_NOMEM : hip_fail(e);
  }
  return src ? copy_in(*out, src, bytes, s) : FR_OK;
}

namespace fr {

void SlotRuns::add(uint32_t unit, uint64_t bytes, uint32_t flag) {
  const uint64_t ns = (bytes + sl - 1) / sl;
  if (ns == 0) return;
  base.push_back((uint64_t(unit) << 32) | flag);
  first.push_back(first.back() + ns);
}

}  // namespace fr

namespace {

// Allocates the slot table of `r` on the device and expands it there: the
// host uploads one (first slot, base) pair per run instead of every slot.
int upload_walk(const SlotRuns& r, fr_plan::Walk& w, const Staging& st) {
  w.sl = r.sl;
  w.t.n = r.n();
  w.t.stride = r.stride();
  int rc = upload(nullptr, 8 * r.stride() * sizeof(uint64_t), (void**)&w.mem, st.s);
  w.t.d = w.mem;
  if (rc != FR_OK || !w.mem) return rc;
  const uint64_t n_runs = r.base.size();
  if (2 * n_runs + 1 > st.runs_cap) return FR_E_RANGE;  // not reached: one run per chunk at most
  uint64_t* d_first = st.runs;
  uint64_t* d_base = d_first + n_runs + 1;
  hipError_t e = hipMemcpyAsync(d_first, r.first.data(), (n_runs + 1) * sizeof(uint64_t),
                                hipMemcpyHostToDevice, st.s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(d_base, r.base.data(), n_runs * sizeof(uint64_t), hipMemcpyHostToDevice,
                       st.s);
  if (e == hipSuccess)
    e = hipError_t(launch_expand_slots(d_first, d_base, n_runs, r.n(), r.stride(), w.mem, st.s));
  if (e == hipSuccess) e = hipStreamSynchronize(st.s);
  return e == hipSuccess ? FR_OK : hip_fail(e);
}

}  // namespace

extern "C" int fr_plan_destroy(fr_plan* p) {
  if (!p) return FR_OK;
  int prev = -1;
  bool switched = false;
  if (p->device >= 0 && hipGetDevice(&prev) == hipSuccess && prev != p->device) {
    switched = hipSetDevice(p->device) == hipSuccess;
  }
  if (p->d_units) (void)hipFree(p->d_units);
  for (auto& w : p->src_walks)
    if (w.mem) (void)hipFree(w.mem);
  if (p->unpack_walk.mem) (void)hipFree(p->unpack_walk.mem);
  if (p->pack_extra.mem) (void)hipFree(p->pack_extra.mem);
  if (p->d_blocks) (void)hipFree(p->d_blocks);
  if (p->unpack_derived.mem) (void)hipFree(p->unpack_derived.mem);
  if (p->d_ublocks) (void)hipFree(p->d_ublocks);
  if (p->d_derived) (void)hipFree(p->d_derived);
  if (p->d_plain) (void)hipFree(p->d_plain);
  if (p->d_scratch) (void)hipFree(p->d_scratch);
  if (p->delta_ids_copied) (void)hipEventSynchronize(p->delta_ids_copied);
  if (p->d_delta) (void)hipFree(p->d_delta);
  if (p->h_delta_ids) (void)hipHostFree(p->h_delta_ids);
  if (p->delta_ids_copied) (void)hipEventDestroy(p->delta_ids_copied);
  if (switched) (void)hipSetDevice(prev);
  delete p;
  return FR_OK;
}

namespace {

// Launch tuning knobs, read from the environment (defaults measured on
// MI355X): workgroup cap (0 = one workgroup per slice), the tile of each
// operation and its line-aligned walks.
LaunchCfg launch_config() {
  LaunchCfg cfg;
  cfg.max_grid = env_u32("FLASHRESTORE_MAX_GRID", 0);
  cfg.delta_grid = env_u32("FLASHRESTORE_DELTA_GRID", kDefaultDeltaGrid);
  const uint32_t all = env_u32("FLASHRESTORE_TILE", ~0u);  // one tile for every operation
  auto pick = [&](const char* name, uint32_t dflt) {
    return int(env_u32(name, all != ~0u ? all : dflt));
  };
  cfg.tile_pack = pick("FLASHRESTORE_TILE_PACK", uint32_t(kTileAuto));
  cfg.tile_unpack = pick("FLASHRESTORE_TILE_UNPACK", uint32_t(kTileAuto));
  cfg.tile_verify = pick("FLASHRESTORE_TILE_VERIFY", uint32_t(kTileAuto));
  cfg.tile_checksum = pick("FLASHRESTORE_TILE_CHECKSUM", uint32_t(kTileAuto));
  // walks: 0 plain, 1 lines of the arena read (for unpack: of the receiver
  // arena written), 2 payload lines, 3 payload slices, 4 payload blocks
  // (pack and unpack take 1-4; compare and checksum 0 or 1, any nonzero
  // value meaning 1); FLASHRESTORE_LINE sets all four; unset, pack and
  // unpack choose by the table (kLineAuto)
  const uint32_t lall = env_u32("FLASHRESTORE_LINE", ~0u);
  auto lpick = [&](const char* name, int dflt, uint32_t modes) {
    const uint32_t v = env_u32(name, lall);
    if (v == ~0u) return dflt;
    if (v == 0) return 0;
    if (v < 5 && (modes >> v) & 1u) return int(v);
    return (modes >> 1) & 1u ? 1 : 0;  // the operation's nearest mode
  };
  cfg.line_pack = lpick("FLASHRESTORE_LINE_PACK", kDefaultLinePack, 0x1E);
  cfg.line_unpack = lpick("FLASHRESTORE_LINE_UNPACK", kDefaultLineUnpack, 0x1E);
  cfg.absorb_pack = int(env_u32("FLASHRESTORE_ABSORB_PACK", kDefaultAbsorbPack) != 0);
  cfg.absorb_unpack = int(env_u32("FLASHRESTORE_ABSORB_UNPACK", kDefaultAbsorbUnpack) != 0);
  cfg.absorb_verify = int(env_u32("FLASHRESTORE_ABSORB_VERIFY", kDefaultAbsorbVerify) != 0);
  cfg.absorb_checksum = int(env_u32("FLASHRESTORE_ABSORB_CHECKSUM", kDefaultAbsorbChecksum) != 0);
  cfg.line_verify = lpick("FLASHRESTORE_LINE_VERIFY", kDefaultLineVerify, 0x2);
  cfg.buf_pack = int(env_u32("FLASHRESTORE_BUF_PACK", kDefaultBufPack) != 0);
  cfg.buf_unpack = int(env_u32("FLASHRESTORE_BUF_UNPACK", kDefaultBufUnpack) != 0);
  cfg.buf_verify = int(env_u32("FLASHRESTORE_BUF_VERIFY", kDefaultBufVerify) != 0);
  cfg.buf_checksum = int(env_u32("FLASHRESTORE_BUF_CHECKSUM", kDefaultBufChecksum) != 0);
  cfg.order_verify = int(env_u32("FLASHRESTORE_ORDER_VERIFY", kDefaultOrderVerify) != 0);
  cfg.order_checksum = int(env_u32("FLASHRESTORE_ORDER_CHECKSUM", kDefaultOrderChecksum) != 0);
  cfg.line_checksum = lpick("FLASHRESTORE_LINE_CHECKSUM", kDefaultLineChecksum, 0x2);
  return cfg;
}

}  // namespace

// The launch configuration of a plan for chunks of C bytes: the
// environment's, with the tiles left unset chosen by chunk size.
static LaunchCfg plan_launch_config(uint64_t C) {
  LaunchCfg cfg = launch_config();
  auto tile = [&](int t, TileOp op) { return t == kTileAuto ? auto_tile(op, C) : t; };
  cfg.tile_pack = tile(cfg.tile_pack, kOpPack);
  cfg.tile_unpack = tile(cfg.tile_unpack, kOpUnpack);
  cfg.tile_verify = tile(cfg.tile_verify, kOpVerify);
  cfg.tile_checksum = tile(cfg.tile_checksum, kOpChecksum);
  return cfg;
}

namespace {

// One record per global chunk.
std::vector<ChunkRec> chunk_records(const fr_tensor_desc* table, uint32_t n, const Layout& L) {
  const uint64_t C = L.C;
  std::vector<ChunkRec> recs(L.n_chunks);
  for (uint32_t k = 0; k < n; k++) {
    const fr_tensor_desc& d = table[k];
    const uint64_t nb = d.numel * esize(d.dtype);
    const uint64_t nc = L.chunk_base[k + 1] - L.chunk_base[k];
    for (uint64_t j = 0; j < nc; j++) {
      ChunkRec& r = recs[L.chunk_base[k] + j];
      r.src_off = d.src_offset + j * C;
      r.dst_off = d.dst_offset + j * C;
      r.pay_off = L.pay_off[k] == kNoPayload ? kNoPayload : L.pay_off[k] + j * C;
      r.len = uint32_t(std::min<uint64_t>(C, nb - j * C));
      // param chunk j covers master chunks 2j and 2j + 1
      r.master = d.derive_from >= 0 ? uint32_t(L.chunk_base[d.derive_from] + 2 * j) : kNoMaster;
    }
  }
  return recs;
}

// Largest power of two, at most kLeadMod, dividing x.
uint32_t pow2_align(uint64_t x) {
  uint32_t a = 1;
  while (a < kLeadMod && x % (2 * a) == 0) a *= 2;
  return a;
}

// Pack / checksum / compare units: every chunk, in chunk order.  The last
// chunk of each sent entry zero-fills the payload gap up to the next one.
// *src_align / *pay_align: the alignment every chunk's sender (payload)
// offset has, up to kLeadMod.
std::vector<SrcUnit> src_units(const std::vector<ChunkRec>& recs, uint32_t n, const Layout& L,
                               uint32_t* src_align, uint32_t* pay_align) {
  std::vector<SrcUnit> units(recs.size());
  *src_align = *pay_align = kLeadMod;
  for (uint64_t c = 0; c < recs.size(); c++) {
    units[c].src_off = recs[c].src_off;
    units[c].pay_off = recs[c].pay_off;
    units[c].len = recs[c].len;
    units[c].c = uint32_t(c);
    units[c].lead = uint16_t(recs[c].src_off % kLeadMod);
    units[c].plead = recs[c].pay_off == kNoPayload ? 0 : uint16_t(recs[c].pay_off % kLeadMod);
    *src_align = std::min(*src_align, pow2_align(recs[c].src_off));
    if (recs[c].pay_off != kNoPayload) *pay_align = std::min(*pay_align, pow2_align(recs[c].pay_off));
  }
  for (uint32_t k = 0, prev = UINT32_MAX; k < n; k++) {
    if (L.pay_off[k] == kNoPayload || L.chunk_base[k + 1] == L.chunk_base[k]) continue;
    if (prev != UINT32_MAX) {
      SrcUnit& u = units[L.chunk_base[prev + 1] - 1];
      u.gap_v = uint32_t((L.pay_off[k] - align16(u.pay_off + u.len)) >> 4);
    }
    prev = k;
  }
  return units;
}

// Unpack units: a derived group per parameter chunk of a derived entry (its
// master chunks travel in it), a plain unit per chunk of every other entry
// that is not such a master.  is_master[k]: entry k feeds a derived entry.
void unpack_units(const fr_tensor_desc* table, uint32_t n, const Layout& L,
                  const std::vector<ChunkRec>& recs, const std::vector<uint8_t>& is_master,
                  std::vector<DerivedUnit>* derived, std::vector<PlainUnit>* plain) {
  for (uint32_t k = 0; k < n; k++) {
    const uint64_t c0 = L.chunk_base[k], c1 = L.chunk_base[k + 1];
    if (table[k].derive_from >= 0) {
      for (uint64_t c = c0; c < c1; c++) {
        const ChunkRec& r = recs[c];
        const ChunkRec& m = recs[r.master];
        DerivedUnit u{};
        u.m_pay_off = m.pay_off;
        u.m_dst_off = m.dst_off;
        u.p_dst_off = r.dst_off;
        u.len = r.len;
        u.m0 = r.master;
        u.c = uint32_t(c);
        derived->push_back(u);
      }
    } else if (!is_master[k]) {
      for (uint64_t c = c0; c < c1; c++) {
        PlainUnit u{};
        u.pay_off = recs[c].pay_off;
        u.dst_off = recs[c].dst_off;
        u.len = recs[c].len;
        u.c = uint32_t(c);
        u.plead = uint32_t(recs[c].pay_off % kLeadMod);
        u.dlead = uint32_t(recs[c].dst_off % kLeadMod);
        plain->push_back(u);
      }
    }
  }
}

// Walks of pack / checksum / compare: every chunk once, one table per slice
// size, alignment, lead handling and order their configurations use (a
// line-aligned walk is the plain one when every chunk starts on a line).
// Pack walks in chunk order, which is payload order; the compare, which
// only reads the arenas, walks them in address order by default (the same
// unless the table lists its tensors out of arena order; the checksum
// measured slower that way, see kDefaultOrderVerify).
int build_src_walks(fr_plan* p, const std::vector<SrcUnit>& units, const Staging& st) {
  const Layout& L = p->layout;
  struct Want {
    int tile, line, absorb;
    bool arena;
  };
  for (uint64_t c = 1; c < units.size(); c++)
    p->chunks_in_arena_order = p->chunks_in_arena_order && units[c - 1].src_off <= units[c].src_off;
  const Want walks[] = {
      {p->cfg.tile_pack, p->cfg.line_pack, p->cfg.absorb_pack, false},
      {p->cfg.tile_checksum, p->cfg.line_checksum, p->cfg.absorb_checksum, p->cfg.order_checksum != 0},
      {p->cfg.tile_verify, p->cfg.line_verify, p->cfg.absorb_verify, p->cfg.order_verify != 0}};
  std::vector<uint32_t> by_addr;
  for (const Want& tw : walks) {
    if (&tw == &walks[0] && p->cfg.line_pack == kLineBlocks) continue;  // build_pack_blocks
    const uint32_t sl = slice_bytes(L.C, tw.tile);
    const uint32_t shift = line_walk(p, tw.tile, tw.line);
    const uint32_t absorb = shift && tw.absorb ? 1u : 0u;
    const bool arena = tw.arena && !p->chunks_in_arena_order;
    bool have = false;
    for (const auto& w : p->src_walks)
      have = have || (w.sl == sl && w.t.shift == shift && w.t.absorb == absorb && w.arena_order == arena);
    if (have) continue;
    if (arena && by_addr.empty()) {  // entries by sender offset, each entry's chunks in order
      std::vector<uint32_t> ent(p->table.size());
      for (uint32_t k = 0; k < ent.size(); k++) ent[k] = k;
      std::stable_sort(ent.begin(), ent.end(), [&](uint32_t x, uint32_t y) {
        return p->table[x].src_offset < p->table[y].src_offset;
      });
      by_addr.reserve(units.size());
      for (uint32_t k : ent)
        for (uint64_t c = L.chunk_base[k]; c < L.chunk_base[k + 1]; c++) by_addr.push_back(uint32_t(c));
    }
    SlotRuns b;
    b.sl = sl;
    b.first.reserve(units.size() + 1);
    b.base.reserve(units.size());
    for (uint64_t i = 0; i < units.size(); i++) {
      const uint32_t c = arena ? by_addr[i] : uint32_t(i);
      b.add(c, units[c].len + (absorb ? 0 : lead_bytes(units[c].lead, units[c].plead, shift, sl)), 0);
    }
    p->src_walks.emplace_back();
    const int rc = upload_walk(b, p->src_walks.back(), st);
    p->src_walks.back().t.shift = shift;
    p->src_walks.back().t.absorb = absorb;
    p->src_walks.back().arena_order = arena;
    if (rc != FR_OK) return rc;
  }
  return FR_OK;
}

// Pack by blocks of the payload (PackBlocks): the sent chunks' units in
// payload order, each block's first unit (found on the device), and a plain
// walk of the chunks without payload.
int build_pack_blocks(fr_plan* p, const std::vector<SrcUnit>& units, const Staging& st) {
  const Layout& L = p->layout;
  const uint32_t block_vecs = tile_bytes(p->cfg.tile_pack) / 16;
  std::vector<SrcUnit> pay;
  pay.reserve(L.n_sent_chunks);
  SlotRuns b;
  b.sl = slice_bytes(L.C, p->cfg.tile_pack);
  for (uint64_t c = 0; c < units.size(); c++) {
    if (units[c].pay_off != kNoPayload) pay.push_back(units[c]);
    else b.add(uint32_t(c), units[c].len, 0);
  }
  PackBlocks& pb = p->pack_blocks;
  pb.n_units = pay.size();
  pb.pay_vecs = pay.empty() ? 0 : L.payload_bytes / 16;
  pb.n_blocks = (pb.pay_vecs + block_vecs - 1) / block_vecs;
  pb.stride = (pb.n_blocks + 7) / 8;
  const uint64_t b_units = (pay.size() * sizeof(SrcUnit) + 255) & ~uint64_t(255);
  int rc = upload(nullptr, b_units + 8 * pb.stride * sizeof(uint32_t), &p->d_blocks, st.s);
  if (rc == FR_OK && p->d_blocks) {
    auto* q = static_cast<uint8_t*>(p->d_blocks);
    pb.units = reinterpret_cast<const SrcUnit*>(q);
    pb.first = reinterpret_cast<const uint32_t*>(q + b_units);
    rc = copy_in(q, pay.data(), pay.size() * sizeof(SrcUnit), st.s);
    if (rc == FR_OK) {
      hipError_t e = hipError_t(launch_block_first(&pb.units->pay_off, pb.n_units, pb.n_blocks,
                                                   pb.stride, block_vecs,
                                                   reinterpret_cast<uint32_t*>(q + b_units), st.s));
      if (e == hipSuccess) e = hipStreamSynchronize(st.s);
      if (e != hipSuccess) rc = hip_fail(e);
    }
  }
  if (rc == FR_OK) rc = upload_walk(b, p->pack_extra, st);
  pb.extra = p->pack_extra.t;
  return rc;
}

// Unpack by blocks of the receiver (UnpackBlocks): the plain chunks sorted
// by receiver offset, the receiver tiles that hold some of their bytes with
// the first chunk touching each (XCD-major), and the walk of the derived
// groups in table order (ids into d_derived, as unpack_units lists them).
int build_unpack_blocks(fr_plan* p, const std::vector<ChunkRec>& recs,
                        const std::vector<uint8_t>& is_master, const Staging& st) {
  const Layout& L = p->layout;
  const uint64_t tile_vecs = tile_bytes(p->cfg.tile_unpack) / 16;
  SlotRuns b;
  b.sl = slice_bytes(L.C, p->cfg.tile_unpack);
  uint32_t id = 0;
  std::vector<uint32_t> ent;  // plain entries, by receiver offset (ranges never overlap)
  for (uint32_t k = 0; k < p->table.size(); k++) {
    if (p->table[k].derive_from >= 0) {
      for (uint64_t c = L.chunk_base[k]; c < L.chunk_base[k + 1]; c++)
        b.add(id++, 2 * uint64_t(recs[c].len), kSlotDerived);
    } else if (!is_master[k]) {
      ent.push_back(k);
    }
  }
  std::sort(ent.begin(), ent.end(), [&](uint32_t x, uint32_t y) {
    return p->table[x].dst_offset < p->table[y].dst_offset;
  });
  std::vector<PlainUnit> units;
  units.reserve(L.n_sent_chunks);
  for (uint32_t k : ent) {
    for (uint64_t c = L.chunk_base[k]; c < L.chunk_base[k + 1]; c++) {
      PlainUnit u{};
      u.pay_off = recs[c].pay_off;
      u.dst_off = recs[c].dst_off;
      u.len = recs[c].len;
      u.c = uint32_t(c);
      units.push_back(u);
    }
  }
  // (tile << 32) | first unit touching it, for every tile some unit touches,
  // in receiver order, stored XCD-major: counted, then written
  auto each_tile = [&](auto&& emit) {
    uint64_t last = ~uint64_t(0);
    for (uint64_t u = 0; u < units.size(); u++) {
      const uint64_t v0 = units[u].dst_off / 16, v1 = v0 + (units[u].len + 15) / 16;
      for (uint64_t t = v0 / tile_vecs; t * tile_vecs < v1; t++)
        if (last == ~uint64_t(0) || last < t) {
          emit((t << 32) | u);
          last = t;
        }
    }
  };
  uint64_t n_tiles = 0;
  each_tile([&](uint64_t) { n_tiles++; });
  UnpackBlocks& ub = p->unpack_blocks;
  ub.n_units = units.size();
  ub.n_blocks = n_tiles;
  ub.stride = (ub.n_blocks + 7) / 8;
  std::vector<uint64_t> xcd(8 * ub.stride, 0);
  uint64_t g = 0;
  each_tile([&](uint64_t e) {
    xcd[(g & 7) * ub.stride + (g >> 3)] = e;
    g++;
  });
  const uint64_t b_units = (units.size() * sizeof(PlainUnit) + 255) & ~uint64_t(255);
  int rc = upload(nullptr, b_units + xcd.size() * sizeof(uint64_t), &p->d_ublocks, st.s);
  if (rc == FR_OK && p->d_ublocks) {
    auto* q = static_cast<uint8_t*>(p->d_ublocks);
    ub.units = reinterpret_cast<const PlainUnit*>(q);
    ub.blocks = reinterpret_cast<const uint64_t*>(q + b_units);
    rc = copy_in(q, units.data(), units.size() * sizeof(PlainUnit), st.s);
    if (rc == FR_OK) rc = copy_in(q + b_units, xcd.data(), xcd.size() * sizeof(uint64_t), st.s);
  }
  if (rc == FR_OK) rc = upload_walk(b, p->unpack_derived, st);
  ub.derived = p->unpack_derived.t;
  return rc;
}

// Walk of unpack, in payload (table) order: a derived entry's groups (their
// master bytes) where the entry stands, plain chunks where theirs.
int build_unpack_walk(fr_plan* p, const std::vector<ChunkRec>& recs,
                      const std::vector<uint8_t>& is_master, const Staging& st) {
  const Layout& L = p->layout;
  SlotRuns b;
  b.sl = slice_bytes(L.C, p->cfg.tile_unpack);
  b.first.reserve(L.n_chunks + 1);
  b.base.reserve(L.n_chunks);
  // plain chunks may be cut at lines of the receiver (mode 1) or of the
  // payload (mode 2), or at slice boundaries of the payload (mode 3), with
  // or without their last slice absorbing the lead
  const uint32_t line = line_walk(p, p->cfg.tile_unpack, p->cfg.line_unpack, true);
  const uint32_t absorb = line && p->cfg.absorb_unpack ? 1u : 0u;
  uint32_t id = 0, ip = 0;
  for (uint32_t k = 0; k < p->table.size(); k++) {
    const uint64_t c0 = L.chunk_base[k], c1 = L.chunk_base[k + 1];
    if (p->table[k].derive_from >= 0) {
      for (uint64_t c = c0; c < c1; c++) b.add(id++, 2 * uint64_t(recs[c].len), kSlotDerived);
    } else if (!is_master[k]) {
      for (uint64_t c = c0; c < c1; c++) {
        const uint32_t lead = absorb ? 0
                                     : lead_bytes(uint32_t(recs[c].dst_off % kLeadMod),
                                                  uint32_t(recs[c].pay_off % kLeadMod), line, b.sl);
        b.add(ip++, recs[c].len + lead, 0);
      }
    }
  }
  const int rc = upload_walk(b, p->unpack_walk, st);
  p->unpack_walk.t.shift = line;
  p->unpack_walk.t.absorb = absorb;
  return rc;
}

// Scratch: accumulators for the largest G any configured tile needs, for two
// arenas, and one flag per chunk.  Its accumulators (16 bytes per chunk at
// least, twice) also hold the staged runs of each slot table (at most one
// run per chunk: 16 bytes per run, and 8 more).
int build_scratch(fr_plan* p, Staging* st) {
  const Layout& L = p->layout;
  uint64_t g = 1;
  for (int t : {p->cfg.tile_pack, p->cfg.tile_unpack, p->cfg.tile_verify, p->cfg.tile_checksum})
    g = std::max<uint64_t>(g, accumulators_per_chunk(L.C, t));
  const uint64_t acc_bytes = L.n_chunks * g * sizeof(fr_chunk_sum);
  const uint64_t flag_bytes = (L.n_chunks * 4 + 255) & ~uint64_t(255);
  const int rc = upload(nullptr, 2 * acc_bytes + flag_bytes, &p->d_scratch, st->s);
  if (rc == FR_OK && p->d_scratch) {
    uint8_t* base = static_cast<uint8_t*>(p->d_scratch);
    p->scratch.acc = reinterpret_cast<fr_chunk_sum*>(base);
    p->scratch.acc_b = reinterpret_cast<fr_chunk_sum*>(base + acc_bytes);
    p->scratch.flags = reinterpret_cast<uint32_t*>(base + 2 * acc_bytes);
    st->runs = reinterpret_cast<uint64_t*>(base);
    st->runs_cap = 2 * acc_bytes / sizeof(uint64_t);
  }
  return rc;
}

// Delta lists built on the device: a location record per chunk (what a
// lane needs about its chunk), room for the records of the longest list
// (pack's one per chunk, or unpack's plain and derived ones), the scan state,
// and the staging of a list given on the host (pinned, so that its upload
// is asynchronous; an event marks when the staging may be refilled).
// Allocated once here, so that no delta call allocates.
int build_delta(fr_plan* p, const std::vector<ChunkRec>& recs, const Staging& st) {
  const Layout& L = p->layout;
  const uint64_t nc = L.n_chunks, nb = (nc + kListBlock - 1) / kListBlock, nw = (nc + 31) / 32;
  auto up = [](uint64_t b) { return (b + 255) & ~uint64_t(255); };
  const uint64_t b_loc = up(nc * sizeof(ChunkLoc));
  const uint64_t b_units = up(std::max(nc * sizeof(SrcUnit), L.n_sent_chunks * sizeof(PlainUnit) +
                                                              (nc - L.n_sent_chunks) * sizeof(DerivedUnit)));
  const uint64_t b_agg = up(nb * sizeof(DeltaAgg)), b_pre = up(nb * sizeof(DeltaPre));
  const uint64_t b_counts = 256, b_bits = up(nw * 4), b_ids = up(nc * 4), b_payof = up(nc * 8);
  const uint64_t total = b_loc + b_units + b_agg + b_pre + b_counts + b_bits + b_ids + b_payof + b_ids;
  int rc = upload(nullptr, total, &p->d_delta, st.s);
  if (rc != FR_OK) return rc;
  uint8_t* q = static_cast<uint8_t*>(p->d_delta);
  auto take = [&](uint64_t b) {
    uint8_t* r = q;
    q += b;
    return r;
  };
  p->d_delta_loc = reinterpret_cast<ChunkLoc*>(take(b_loc));
  uint8_t* units = take(b_units);
  p->d_delta_src = reinterpret_cast<SrcUnit*>(units);
  p->d_delta_plain = reinterpret_cast<PlainUnit*>(units);
  p->d_delta_derived = reinterpret_cast<DerivedUnit*>(units + L.n_sent_chunks * sizeof(PlainUnit));
  p->d_delta_agg = reinterpret_cast<DeltaAgg*>(take(b_agg));
  p->d_delta_pre = reinterpret_cast<DeltaPre*>(take(b_pre));
  p->d_delta_counts = reinterpret_cast<uint64_t*>(take(b_counts));
  p->d_delta_bits = reinterpret_cast<uint32_t*>(take(b_bits));
  p->d_delta_ids = reinterpret_cast<uint32_t*>(take(b_ids));
  p->d_delta_payof = reinterpret_cast<uint64_t*>(take(b_payof));
  p->d_delta_m0 = reinterpret_cast<uint32_t*>(take(b_ids));
  std::vector<ChunkLoc> loc(nc);
  std::vector<uint32_t> m0(nc, 0);
  for (uint32_t k = 0; k < p->table.size(); k++) {
    const uint64_t c0 = L.chunk_base[k], c1 = L.chunk_base[k + 1];
    for (uint64_t c = c0; c < c1; c++) {
      const ChunkRec& r = recs[c];
      ChunkLoc& l = loc[c];
      l.src_off = r.src_off;
      l.dst_off = r.dst_off;
      // a derived chunk's master bytes: master chunks 2j and 2j + 1 from chunk 2j on
      l.m_dst_off = r.master == kNoMaster ? 0 : recs[r.master].dst_off;
      l.len = r.len;
      l.flags = (r.master == kNoMaster ? 0u : kLocDerived) | (c == c0 ? kLocFirst : 0u) |
                (c + 1 == c1 ? kLocLast : 0u);
      m0[c] = r.master == kNoMaster ? 0u : r.master;
    }
  }
  rc = copy_in(p->d_delta_loc, loc.data(), nc * sizeof(ChunkLoc), st.s);
  if (rc == FR_OK) rc = copy_in(p->d_delta_m0, m0.data(), nc * sizeof(uint32_t), st.s);
  if (rc != FR_OK) return rc;
  hipError_t e = hipSuccess;
  if (nc)
    e = hipHostMalloc(reinterpret_cast<void**>(&p->h_delta_ids), nc * 4, hipHostMallocDefault);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&p->delta_ids_copied, hipEventDisableTiming);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e == hipErrorOutOfMemory ? FR_E_NOMEM : hip_fail(e);
  }
  return FR_OK;
}

}  // namespace

extern "C" int fr_plan_create_ex(const fr_tensor_desc* table, uint32_t n, uint64_t C,
                                 uint64_t src_bytes, uint64_t dst_bytes, uint64_t seg,
                                 fr_plan** out) {
  if (!out) return FR_E_INVAL;
  fr_plan* p = nullptr;
  try {
    p = new fr_plan();
    int rc = validate_and_layout(table, n, C, seg, src_bytes, dst_bytes, &p->layout);
    if (rc != FR_OK) {
      delete p;
      return rc;
    }
    p->table.assign(table, table + n);
    p->src_arena_bytes = src_bytes;
    p->dst_arena_bytes = dst_bytes;
    int dev = -1;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
      delete p;
      return hip_fail(e);
    }
    p->device = dev;
    p->cfg = plan_launch_config(C);

    const Layout& L = p->layout;
    const std::vector<ChunkRec> recs = chunk_records(table, n, L);
    std::vector<uint8_t> is_master(n, 0);
    for (uint32_t k = 0; k < n; k++)
      if (table[k].derive_from >= 0) is_master[table[k].derive_from] = 1;
    std::vector<DerivedUnit> derived;
    std::vector<PlainUnit> plain;
    unpack_units(table, n, L, recs, is_master, &derived, &plain);
    p->n_derived = uint32_t(derived.size());
    p->n_plain = uint32_t(plain.size());
    for (const PlainUnit& u : plain) p->dst_align = std::min(p->dst_align, pow2_align(u.dst_off));
    const std::vector<SrcUnit> units = src_units(recs, n, L, &p->src_align, &p->pay_align);
    // automatic walks: blocks where chunks of the side written start inside lines
    auto resolve = [](int mode, uint32_t align, int aligned) {
      return mode != kLineAuto ? mode : align < kLine ? kLineBlocks : aligned;
    };
    p->cfg.line_pack = resolve(p->cfg.line_pack, p->pay_align, kAlignedLinePack);
    p->cfg.line_unpack = resolve(p->cfg.line_unpack, p->dst_align, kAlignedLineUnpack);

    Staging st;
    const hipError_t es = hipStreamCreateWithFlags(&st.s, hipStreamNonBlocking);
    if (es != hipSuccess) {
      st.s = nullptr;
      delete p;
      return hip_fail(es);
    }
    rc = build_scratch(p, &st);
    if (rc == FR_OK)
      rc = upload(units.data(), units.size() * sizeof(SrcUnit), (void**)&p->d_units, st.s);
    if (rc == FR_OK) rc = build_src_walks(p, units, st);
    if (rc == FR_OK && p->cfg.line_pack == kLineBlocks) rc = build_pack_blocks(p, units, st);
    if (rc == FR_OK && p->cfg.line_unpack != kLineBlocks) rc = build_unpack_walk(p, recs, is_master, st);
    if (rc == FR_OK && p->cfg.line_unpack == kLineBlocks) rc = build_unpack_blocks(p, recs, is_master, st);
    if (rc == FR_OK)
      rc = upload(derived.data(), derived.size() * sizeof(DerivedUnit), (void**)&p->d_derived,
                  st.s);
    if (rc == FR_OK)
      rc = upload(plain.data(), plain.size() * sizeof(PlainUnit), (void**)&p->d_plain, st.s);
    if (rc == FR_OK) rc = build_delta(p, recs, st);
    if (rc != FR_OK) {
      fr_plan_destroy(p);
      return rc;
    }
  } catch (const std::bad_alloc&) {
    if (p) fr_plan_destroy(p);
    return FR_E_NOMEM;
  }
  *out = p;
  return FR_OK;
}

extern "C" int fr_plan_create(const fr_tensor_desc* table, uint32_t n, uint64_t C,
                              uint64_t src_bytes, uint64_t dst_bytes, fr_plan** out) {
  return fr_plan_create_ex(table, n, C, src_bytes, dst_bytes, kDefaultSegmentAlign, out);
}

extern "C" int fr_plan_get_info(const fr_plan* p, fr_plan_info* info) {
  if (!p || !info) return FR_E_INVAL;
  // the walks the operations take (a line-aligned mode is the plain walk
  // where every chunk of its side starts on a line)
  const LaunchCfg& c = p->cfg;
  const uint32_t pw = c.line_pack == kLineBlocks ? uint32_t(kLineBlocks)
                                                 : line_walk(p, c.tile_pack, c.line_pack);
  const uint32_t uw = c.line_unpack == kLineBlocks ? uint32_t(kLineBlocks)
                                                   : line_walk(p, c.tile_unpack, c.line_unpack, true);
  fill_info(p->layout, uint32_t(p->table.size()), p->src_arena_bytes, p->dst_arena_bytes,
            p->device, c, info, pw, uw);
  return FR_OK;
}

extern "C" int fr_plan_chunk_of(const fr_plan* p, uint32_t entry, uint64_t byte, uint64_t* chunk) {
  if (!p || !chunk) return FR_E_INVAL;
  if (entry >= p->table.size()) return FR_E_RANGE;
  const fr_tensor_desc& d = p->table[entry];
  uint64_t nb = d.numel * (d.dtype == FR_F32 ? 4 : 2);
  if (byte >= nb) return FR_E_RANGE;
  *chunk = p->layout.chunk_base[entry] + byte / p->layout.C;
  return FR_OK;
}

extern "C" int fr_plan_entry_layout(const fr_plan* p, uint32_t entry, uint64_t* payload_offset,
                                    uint64_t* first_chunk, uint64_t* n_chunks) {
  if (!p) return FR_E_INVAL;
  if (entry >= p->table.size()) return FR_E_RANGE;
  if (payload_offset) *payload_offset = p->layout.pay_off[entry];
  if (first_chunk) *first_chunk = p->layout.chunk_base[entry];
  if (n_chunks) *n_chunks = p->layout.chunk_base[entry + 1] - p->layout.chunk_base[entry];
  return FR_OK;
}
