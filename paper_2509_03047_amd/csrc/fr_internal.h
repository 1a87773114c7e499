// Internal declarations shared by the host sources and the gfx950 kernels.
#pragma once

#include <stdint.h>

#include <vector>

#include "flashrestore.h"

namespace fr {

constexpr uint64_t kNoPayload = ~uint64_t(0);
// A payload segment (an entry, or a run of consecutive chunks of a delta
// list) starts at a multiple of the plan's segment alignment: 16 by default
// (segments back to back), up to kMaxSegmentAlign.  With 4096 the slices of
// a segment start at 4 KiB boundaries of the payload, which on MI355X makes
// pack up to a fifth faster on tables of many small or oddly placed tensors.
constexpr uint64_t kDefaultSegmentAlign = 16;
constexpr uint64_t kMaxSegmentAlign = uint64_t(1) << 20;
constexpr uint32_t kNoMaster = 0xFFFFFFFFu;
constexpr uint32_t kLine = 128;  // L2 cache line (bytes)
// Unit records keep offsets modulo this, enough for any slice size (at most
// 16 KiB), so that a walk can cut slices at lines or at slice boundaries.
constexpr uint32_t kLeadMod = 32768;
// Bytes of the static device array the no-allocation calls use as scratch
// (kernels.hip); the public limit FR_STATIC_SCRATCH_BYTES.
constexpr uint64_t kStaticScratchBytes = FR_STATIC_SCRATCH_BYTES;

// One record per global chunk id (host side; the device tables are built
// from these).
struct alignas(16) ChunkRec {
  uint64_t src_off;  // chunk start in the sender / replica arena
  uint64_t pay_off;  // chunk start in the payload; kNoPayload for derived entries
  uint64_t dst_off;  // chunk start in the receiver arena
  uint32_t len;      // bytes in this chunk (<= C, even)
  uint32_t master;   // derived chunk j: global id of master chunk 2j; else kNoMaster
};
static_assert(sizeof(ChunkRec) == 32, "ChunkRec is 32 bytes");

// Device unit records.  A workgroup reads its slot (see SlotTable), then the
// record of the unit it works on, with uniform (scalar) loads, and needs
// nothing else to address its data.

// Unit of pack, checksum and replica compare: one chunk of the sender (or
// replica) arena.
struct alignas(16) SrcUnit {
  uint64_t src_off;  // chunk start in the sender / replica arena
  uint64_t pay_off;  // chunk start in the payload; kNoPayload: read and summed only
  uint32_t len;      // bytes in this chunk (<= C, even)
  uint32_t c;        // its sums slot: global chunk id, or list position for a delta
  uint32_t gap_v;    // zero vectors pack writes after the chunk's 16-byte-padded end
                     //   (the gap up to the next segment; < segment alignment / 16)
  uint16_t lead;     // src_off mod kLeadMod: where the chunk starts within lines / slices
  uint16_t plead;    // pay_off mod kLeadMod (0 without payload): the same in the payload
};
static_assert(sizeof(SrcUnit) == 32, "SrcUnit is 32 bytes");

// Unpack units.
// A derived group: bf16 parameter chunk j and the fp32 master chunks 2j and
// 2j + 1 it is rounded from.
struct alignas(16) DerivedUnit {
  uint64_t m_pay_off;  // payload offset of master chunk 2j (the group's first master byte)
  uint64_t m_dst_off;  // receiver offset of master chunk 2j
  uint64_t p_dst_off;  // receiver offset of parameter chunk j
  uint32_t len;        // parameter chunk bytes L (the group holds 2L master bytes)
  uint32_t m0;         // global id of master chunk 2j
  uint32_t c;          // global id of parameter chunk j
  uint32_t pad_;
};
static_assert(sizeof(DerivedUnit) == 48, "DerivedUnit is 48 bytes");

// A chunk copied as it is.
struct alignas(16) PlainUnit {
  uint64_t pay_off;
  uint64_t dst_off;
  uint32_t len;
  uint32_t c;
  uint32_t plead;  // pay_off mod kLeadMod
  uint32_t dlead;  // dst_off mod kLeadMod
};
static_assert(sizeof(PlainUnit) == 32, "PlainUnit is 32 bytes");

// A walk: one 64-bit slot per workgroup id, (unit << 32) | j with j the
// slice of that unit, bytes [j * SL, (j + 1) * SL) of it (for unpack,
// kSlotDerived in the low word marks a derived group).  Units are listed in
// address order and a unit of b bytes has ceil(b / SL) slots, so no
// workgroup of a launch is idle.  (Giving every unit C / SL slots instead
// leaves the slots past a short chunk's end idle: a few thousand idle
// workgroups among two million cost 4 % of the bandwidth, and moving the
// short chunks to the end of the launch costs as much, since they are then
// read scattered.)  The table is stored XCD-major: the
// dispatcher hands workgroup g to XCD g mod 8, and slot g sits at
// (g mod 8) * stride + g / 8, so each XCD reads its own slots contiguously.
constexpr uint32_t kSlotDerived = 0x80000000u;

struct SlotTable {
  const uint64_t* d = nullptr;  // NULL: implicit walk (below)
  uint64_t n = 0;       // slots (workgroups to launch)
  uint64_t stride = 0;  // ceil(n / 8); the table holds 8 * stride entries
  // Implicit walk, for the scattered chunk lists of a delta call, which
  // would gain nothing from a table: every unit has 2^implicit_shift slots
  // and slot g is (g >> implicit_shift, g mod 2^implicit_shift); slots past
  // a short unit's end do nothing.
  uint32_t implicit_shift = 0;
  // Line-aligned walk (SrcUnit walks only): slice j of a chunk covers chunk
  // bytes [j SL - lead, (j + 1) SL - lead), so every cut between slices falls
  // on a cache-line boundary and no line is fetched or written by two
  // workgroups; a chunk has ceil((lead + len) / SL) slices (one more than a
  // plain walk's when it starts inside a line and ends near a slice end).
  // shift 1 takes lead as the offset into a line of the arena read
  // (SrcUnit::lead), 2 into a line of the payload (SrcUnit::plead); 3 cuts
  // at multiples of SL in the payload instead of lines (lead = the payload
  // offset mod SL; for pack's SrcUnit walks and unpack's plain chunks).
  uint32_t shift = 0;
  // With absorb, a unit keeps the plain walk's ceil(len / SL) slices and its
  // last slice also takes the leftover lead bytes (at most a line less 16
  // bytes for modes 1 and 2) instead of a further, nearly empty, slice.
  uint32_t absorb = 0;
  // Implicit walk over a list built on the device: n covers the longest
  // list, and only the slots of the first *count units work.
  const uint64_t* count = nullptr;
};

// A slot table as runs, built on the host (plan.cpp) and expanded on the
// device (launch_expand_slots): run r holds the slots base[r] | 0,
// base[r] | 1, ..., base[r] | (first[r + 1] - first[r] - 1), runs in walk
// order, none empty.
struct SlotRuns {
  std::vector<uint64_t> first{0};  // n_runs + 1 entries: prefix of slot counts
  std::vector<uint64_t> base;      // n_runs entries: (unit << 32) | flag
  uint32_t sl = 0;                 // slice bytes
  void add(uint32_t unit, uint64_t bytes, uint32_t flag);  // ceil(bytes / sl) slots
  uint64_t n() const { return first.back(); }
  uint64_t stride() const { return (n() + 7) / 8; }
};

// Host-side layout of a validated table.
struct Layout {
  uint64_t C = 0;
  uint64_t seg = 0;  // payload segment alignment
  uint64_t n_chunks = 0;
  uint64_t payload_bytes = 0;
  uint64_t state_bytes = 0;
  uint64_t n_sent_chunks = 0;       // chunks of non-derived entries
  uint64_t delta_payload_max = 0;   // the largest delta payload any list of chunks can need
  std::vector<uint64_t> pay_off;     // per entry; kNoPayload for derived
  std::vector<uint64_t> chunk_base;  // n_entries + 1
};

int validate_and_layout(const fr_tensor_desc* table, uint32_t n, uint64_t C, uint64_t seg,
                        uint64_t src_bytes, uint64_t dst_bytes, Layout* out);

// Launch configuration of a plan.  A tile is B threads x U 16-byte vectors
// per workgroup: 0 = 256x1, 1 = 512x1, 2 = 256x2, 3 = 256x4, 4 = 64x4,
// 5 = 128x2, 6 = 64x2, 7 = 64x1, 8 = 128x1, 9 = 128x4, 10 = 64x8.
struct LaunchCfg {
  uint32_t max_grid = 0;  // cap on workgroups per launch (0: hardware limit); grid-stride beyond
  uint32_t delta_grid = 0;  // cap on workgroups walking a list built on the device (0: none)
  int tile_pack = 0, tile_unpack = 0, tile_verify = 0, tile_checksum = 0;
  // line-aligned walks (SlotTable::shift) per operation: 0 off, 1 cut at
  // lines of the arena read, 2 (pack) at lines of the payload, 3 (pack,
  // unpack) at slice boundaries of the payload; pack 4: by blocks of the
  // payload (PackBlocks) instead of slices of chunks
  int line_pack = 0, line_unpack = 0, line_verify = 0, line_checksum = 0;
  // line-aligned walks whose units' last slice absorbs the lead
  int absorb_pack = 0, absorb_unpack = 0, absorb_verify = 0, absorb_checksum = 0;
  // slices loaded through buffer resources (every load of a thread in
  // flight at once) rather than predicated global loads
  int buf_pack = 0, buf_unpack = 0, buf_verify = 0, buf_checksum = 0;
  // the compare's and the checksum's walks in arena address order rather
  // than chunk order (they differ when a table lists tensors out of arena order)
  int order_verify = 0, order_checksum = 0;
};

// Device scratch owned by a plan: per-chunk accumulators (G per chunk, see
// accumulators_per_chunk), a second set for the replica compare's sums of
// arena B, and one 32-bit flag per chunk.  Every operation clears what it
// uses first, so operations on one plan must not overlap in time.
struct Scratch {
  fr_chunk_sum* acc = nullptr;
  fr_chunk_sum* acc_b = nullptr;
  uint32_t* flags = nullptr;
};

struct UnpackArgs {
  const DerivedUnit* derived;
  uint32_t n_derived;
  const PlainUnit* plain;
  uint32_t n_plain;
  SlotTable slots;  // derived groups and plain chunks in payload order
  uint32_t n_chunks;
  uint64_t C;
  const void* payload;
  const fr_chunk_sum* sums;
  void* dst;
  uint32_t* bitmap;
  uint64_t* n_bad;
  Scratch scratch;
};

// A delta restore (a list of chunks) on the receiver: sent chunks first,
// then derived chunks recomputed from the receiver's masters.
struct UnpackDeltaArgs {
  const PlainUnit* plain;      // sent chunks; c = list position
  uint32_t n_plain;
  const DerivedUnit* derived;  // derived chunks; m_pay_off = master's receiver offset, c = list position
  uint32_t n_derived;
  SlotTable plain_slots, derived_slots;
  uint32_t n_ids;
  uint64_t C;
  const void* payload;
  const fr_chunk_sum* sums;    // n_ids, list order
  void* dst;
  uint32_t* bitmap;
  uint64_t* n_bad;
  Scratch scratch;
  const uint64_t* live = nullptr;  // list built on the device: its length (n_ids is the bound)
  const uint32_t* bad = nullptr;   // per list position: 1 = flag it whatever its sums
  // the list (bit c set = chunk c listed) and each listed sent chunk's
  // payload offset (DeltaBuild::pay_of): a derived chunk reads a master
  // chunk from the payload when it was re-sent, else from the receiver
  const uint32_t* bits = nullptr;
  const uint64_t* pay_of = nullptr;
};

// Where a chunk lives, for lists of chunks built on the device: one record
// per chunk id, so that a lane finds everything about its chunk with one load.
constexpr uint32_t kLocDerived = 1;  // a bf16 parameter re-derived from its master
constexpr uint32_t kLocFirst = 2;    // the first chunk of its entry
constexpr uint32_t kLocLast = 4;     // the last chunk of its entry
struct alignas(16) ChunkLoc {
  uint64_t src_off;    // in the sender / replica arena
  uint64_t dst_off;    // in the receiver arena
  uint64_t m_dst_off;  // derived: receiver offset of the master bytes it is rounded from
  uint32_t len;        // bytes
  uint32_t flags;      // kLoc*
};
static_assert(sizeof(ChunkLoc) == 32, "ChunkLoc is 32 bytes");

// Scan element of a delta list: the map x -> x + q (has = 0) or
// x -> align_A(x + p) + q (has = 1) of the payload end over some chunks,
// with their counts of sent (ns) and derived (nd) chunks.
struct DeltaAgg {
  uint32_t ns, nd, has, pad_;
  uint64_t p, q;
};
// Before a block of chunks: the payload end and the counts.
struct DeltaPre {
  uint64_t end;
  uint32_t ns, nd;
};
// Totals of a list built on the device (plan-owned device words).
enum DeltaCount { kDeltaIds = 0, kDeltaSent = 1, kDeltaDerived = 2, kDeltaEnd = 3 };
// Chunks per block of the list builder (one lane each).
constexpr uint32_t kListBlock = 256;

struct DeltaBuild {
  const ChunkLoc* loc;       // per chunk id
  const uint32_t* bits;      // the list: bit c set = chunk c listed
  uint64_t n_chunks;         // the plan's chunks (bits past them are ignored)
  uint64_t seg;              // payload segment alignment A
  DeltaAgg* agg;             // per block of kListBlock chunks
  DeltaPre* pre;             // per block
  uint64_t* counts;          // [kDeltaIds, kDeltaSent, kDeltaDerived, kDeltaEnd]
  uint64_t* user_counts;     // NULL or the caller's [list length, payload bytes]
  SrcUnit* src_units;        // pack: one per listed chunk, list order
  PlainUnit* plain;          // unpack: sent chunks
  DerivedUnit* derived;      // unpack: derived chunks (re-derived from the receiver's masters)
  uint32_t* bad;             // unpack: per list position, 1 = beyond the readable payload
  uint64_t* pay_of;          // unpack: per chunk id, a listed sent chunk's payload offset
                             //   (kNoPayload if beyond the readable payload)
  const uint32_t* m0;        // per chunk id: a derived chunk's first master chunk
  uint64_t payload_limit;    // pack: payload capacity; unpack: readable payload bytes
  fr_chunk_sum* acc;         // accumulators of the operation, cleared per listed position
  uint32_t acc_shift;        // log2 of the accumulators per list position
  uint64_t* zero_word;       // NULL, or a counter the operation starts from 0 (n_bad)
};

// Bytes of one slice for a tile, and the accumulators a chunk of C bytes
// needs with that tile (kernels.hip).
uint32_t tile_bytes(int tile);
inline uint32_t slice_bytes(uint64_t C, int tile) {
  const uint32_t t = tile_bytes(tile);
  return C < t ? uint32_t(C) : t;
}
uint64_t accumulators_per_chunk(uint64_t C, int tile);

// The line-aligned mode an operation with this tile and line setting walks
// in: the setting when some chunk starts inside a line of the side it keys
// on (mode 1: the arena the operation reads, or with `receiver` unpack's
// receiver arena) and a slice spans at least two lines, else 0 (the plain
// walk is then the same thing).
inline uint32_t line_walk(const fr_plan* p, int tile, int line, bool receiver = false);
inline uint32_t lead_bytes(uint32_t lead, uint32_t plead, uint32_t line, uint32_t sl);

// Pack walked by blocks of the payload, one tile (T = B U vectors) per
// workgroup across chunk boundaries, plus a slot walk over the chunks that
// have no payload (launch_pack_blocks).
struct PackBlocks {
  const SrcUnit* units = nullptr;   // sent chunks in payload order (c = global chunk id)
  const uint32_t* first = nullptr;  // per block, XCD-major: the unit holding its first vector
  uint64_t n_units = 0, n_blocks = 0, stride = 0, pay_vecs = 0;
  SlotTable extra{};  // the chunks without payload, ids into the plan's d_units
};
// Pack walked by blocks of the payload, unpack by blocks of the receiver
// arena (tiles of the side written).
constexpr int kLineBlocks = 4;
// Blocks where chunks of the side written start inside lines, else the
// operation's line walk.
constexpr int kLineAuto = -1;
// A tile chosen by the chunk size at plan creation (no tile variable set).
constexpr int kTileAuto = -1;

// Unpack walked by blocks of the receiver arena: the plain chunks in
// receiver order, the tiles that hold some of their bytes, and the walk of
// the derived groups (launch_unpack_blocks).
struct UnpackBlocks {
  const PlainUnit* units = nullptr;
  const uint64_t* blocks = nullptr;  // XCD-major: (tile index << 32) | first unit in it
  uint64_t n_units = 0, n_blocks = 0, stride = 0;
  SlotTable derived{};  // derived groups only, ids into the plan's d_derived
};

// Kernel launchers (kernels.hip).  They assume validated arguments, enqueue
// on `stream` and return the hipError_t of the launches as an int.
// `units` holds n_chunks records whose sums slots c cover [0, n_chunks);
// `slots` walks them at the slice size of the operation's tile.
int launch_pack(const SrcUnit* units, const SlotTable& slots, uint32_t n_chunks, uint64_t C,
                const void* src, void* payload, fr_chunk_sum* sums, const Scratch& scr,
                const LaunchCfg& cfg, void* stream);
int launch_pack_blocks(const SrcUnit* units, const PackBlocks& pb, uint32_t n_chunks, uint64_t C,
                       const void* src, void* payload, fr_chunk_sum* sums, const Scratch& scr,
                       const LaunchCfg& cfg, void* stream);
// out[0 .. 8 * stride) <- the first unit of every block of block_vecs
// vectors (PackBlocks::first), for units whose payload offsets are
// pay_off[0], pay_off[4], ... (32-byte records).
int launch_block_first(const uint64_t* pay_off, uint64_t n_units, uint64_t n_blocks,
                       uint64_t stride, uint32_t block_vecs, uint32_t* out, void* stream);
int launch_unpack_blocks(const UnpackArgs& args, const UnpackBlocks& ub, const LaunchCfg& cfg,
                         void* stream);
int launch_checksum(const SrcUnit* units, const SlotTable& slots, uint32_t n_chunks, uint64_t C,
                    const void* base, fr_chunk_sum* sums, const Scratch& scr,
                    const LaunchCfg& cfg, void* stream);
int launch_unpack(const UnpackArgs& args, const LaunchCfg& cfg, void* stream);
int launch_unpack_delta(const UnpackDeltaArgs& args, const LaunchCfg& cfg, void* stream);
int launch_verify(const SrcUnit* units, const SlotTable& slots, uint32_t n_chunks, uint64_t C,
                  const void* a, const void* b, uint32_t* bitmap, uint64_t* n_diff,
                  fr_chunk_sum* sums_a, fr_chunk_sum* sums_b, const Scratch& scr,
                  const LaunchCfg& cfg, void* stream);
// Bit c of `bitmap` set iff the two sums of chunk c differ; `count` the bits set.
int launch_compare_sums(const fr_chunk_sum* a, const fr_chunk_sum* b, uint32_t n_chunks,
                        uint32_t* bitmap, uint64_t* count, void* stream);
// The unit records of a delta list given as a bitmap, built on the device:
// pack's SrcUnit list, or unpack's plain and derived lists, and the counts;
// it also clears the accumulators of the listed positions and *zero_word,
// so the operation's own launches need not.
int launch_delta_build(const DeltaBuild& b, bool for_pack, void* stream);
// bits[0 .. words) <- the bitmap of ids[0 .. n) (ids < 32 * words).
int launch_ids_to_bits(const uint32_t* ids, uint64_t n, uint32_t* bits, uint64_t words,
                       void* stream);
// Device address of the static scratch array (kStaticScratchBytes, 256-byte
// aligned) on `device`, which must be the current device; resolved on the
// first call per device.  Returns a hipError_t as an int.
int static_scratch_address(int device, void** out);
// Writes the XCD-major image (8 * stride entries, zero past slot n - 1) of
// the slot table whose runs are first[0 .. n_runs] and base[0 .. n_runs - 1]
// (device arrays; first[0] = 0, first[n_runs] = n, no empty run).
int launch_expand_slots(const uint64_t* first, const uint64_t* base, uint64_t n_runs, uint64_t n,
                        uint64_t stride, uint64_t* out, void* stream);

}  // namespace fr

struct fr_plan {
  int device = -1;
  std::vector<fr_tensor_desc> table;
  fr::Layout layout;
  uint64_t src_arena_bytes = 0, dst_arena_bytes = 0;
  fr::SrcUnit* d_units = nullptr;    // n_chunks records, chunk order
  // slot tables of the walks: pack / checksum / compare (one per slice size
  // their tiles use) and unpack
  struct Walk {
    uint32_t sl = 0;
    fr::SlotTable t{};  // t.shift: the line-aligned mode (0 off, 1 arena lines, 2 payload lines)
    uint64_t* mem = nullptr;
    bool arena_order = false;  // units in arena address order rather than chunk (payload) order
  };
  bool chunks_in_arena_order = true;  // chunk order is already arena address order
  uint32_t dst_align = fr::kLeadMod;     // the same for every plain unpack chunk's receiver offset
  uint32_t src_align = fr::kLeadMod;   // largest power of two (<= kLeadMod) dividing every chunk's src_off
  uint32_t pay_align = fr::kLeadMod;   // the same for every sent chunk's payload offset
  std::vector<Walk> src_walks;
  Walk unpack_walk;
  // pack / unpack by payload blocks (cfg.line_* == kLineBlocks): the sent
  // chunks' units in payload order and each block's first unit (one
  // allocation each), and the walk of the rest (pack: the chunks without
  // payload; unpack: the derived groups)
  void* d_blocks = nullptr;
  fr::PackBlocks pack_blocks{};
  Walk pack_extra;
  void* d_ublocks = nullptr;
  fr::UnpackBlocks unpack_blocks{};
  Walk unpack_derived;
  fr::DerivedUnit* d_derived = nullptr;  // unpack units: derived groups
  uint32_t n_derived = 0;
  fr::PlainUnit* d_plain = nullptr;      // unpack units: plain chunks
  uint32_t n_plain = 0;
  void* d_scratch = nullptr;         // one allocation holding `scratch`
  // Delta lists, built on the device (one allocation, carved at creation):
  void* d_delta = nullptr;
  fr::ChunkLoc* d_delta_loc = nullptr;  // per chunk id
  fr::SrcUnit* d_delta_src = nullptr; // pack records; shares its bytes with the two below
  fr::PlainUnit* d_delta_plain = nullptr;
  fr::DerivedUnit* d_delta_derived = nullptr;
  fr::DeltaAgg* d_delta_agg = nullptr;
  fr::DeltaPre* d_delta_pre = nullptr;
  uint64_t* d_delta_counts = nullptr;  // fr::DeltaCount
  uint32_t* d_delta_bits = nullptr;    // bitmap of a host list
  uint32_t* d_delta_ids = nullptr;     // a host list, uploaded
  uint64_t* d_delta_payof = nullptr;   // per chunk: payload offset in the last delta unpack
  uint32_t* d_delta_m0 = nullptr;      // per chunk: a derived chunk's first master chunk
  uint32_t* h_delta_ids = nullptr;     // pinned staging of a host list
  hipEvent_t delta_ids_copied = nullptr;  // the last upload from the staging has completed
  fr::Scratch scratch{};
  fr::LaunchCfg cfg{};
};

inline uint32_t fr::line_walk(const fr_plan* p, int tile, int line, bool receiver) {
  const uint32_t sl = slice_bytes(p->layout.C, tile);
  const uint32_t grain = line == 1 || line == 2 ? kLine : line == 3 ? sl : 0;
  const uint32_t align = line == 1 ? (receiver ? p->dst_align : p->src_align) : p->pay_align;
  return grain && align < grain && sl >= 2 * kLine ? uint32_t(line) : 0u;
}

// Bytes a walk of mode `line` starts a unit early: its offset into a line,
// or into a slice of `sl` bytes (mode 3); 0 for a plain walk.
inline uint32_t fr::lead_bytes(uint32_t lead, uint32_t plead, uint32_t line, uint32_t sl) {
  return line == 1 ? lead % kLine : line == 2 ? plead % kLine : line == 3 ? plead % sl : 0u;
}
