/*
 * flashrestore: data-parallel replica state restore on MI355X (gfx950).
 *
 * The checkpoint-free recovery of FlashRecovery (arXiv 2509.03047) rebuilds a
 * recreated process's model state -- parameters, optimizer state and other
 * training state -- from a healthy replica in its data-parallel group rather
 * than from a checkpoint, by collective communication (Section III-B item 3;
 * Section III-E, its part on restoring the model states).  Data parallelism is what makes
 * the replicas exist and keeps them identical (Section III-A).  This library
 * is the per-GPU data path of that restore:
 *
 *   fr_pack_state      donor side: gather every tensor of the state into one
 *                      contiguous transfer buffer and checksum every chunk;
 *   fr_unpack_state    receiver side: scatter the buffer into the receiver's
 *                      tensor layout, re-derive bf16 parameters from their
 *                      fp32 master copies, and check every chunk;
 *   fr_verify_replicas compare two replicas chunk by chunk;
 *   fr_checksum_state  chunk checksums of one state.
 *
 * The transfer itself (the collective) is not part of this library: between
 * pack and unpack the caller moves `payload` and `sums` by any means.  The
 * paper fixes no buffer format, checksum or dtype handling; the definitions
 * below are this library's and are stated in full so that any other
 * implementation can reproduce every output byte.
 *
 * Definitions
 *   Tensor table.  An array of fr_tensor_desc.  Entry k has
 *     nbytes_k = numel_k * esize (4 for FR_F32, 2 for FR_BF16).
 *   Chunks.  Entry k is cut into ceil(nbytes_k / C) chunks of C = chunk_bytes
 *     bytes (only the last may be shorter).  Chunk j of entry k has global id
 *     chunk_base_k + j, where chunk_base is the exclusive prefix sum of the
 *     per-entry chunk counts in table order.  Derived entries are chunked the
 *     same way.
 *   FRSUM-128.  A chunk's bytes read as little-endian 32-bit words w_0, w_1,
 *     ... (a short last word is zero-filled): sum = sum_i w_i mod 2^64 and
 *     wsum = sum_i (i+1) w_i mod 2^64.  Any single-bit change alters sum; any
 *     two-bit change within a chunk of < 2^32 words alters (sum, wsum).
 *   Derived entries.  A FR_BF16 entry with derive_from = s >= 0 holds
 *     RNE(master_s): it is not sent; its chunk sums are.  The receiver
 *     recomputes it from the received master, so the check proves it equal to
 *     the donor's bytes.
 *   RNE.  fp32 bit pattern u -> bf16: if (u & 0x7FFFFFFF) > 0x7F800000 (NaN)
 *     the result is (u >> 16) | 0x0040, otherwise the nearer bf16 neighbour
 *     with ties to an even last bit, overflow to infinity, denormals rounded
 *     exactly (no flush to zero).
 *   Payload.  The bytes of every non-derived entry in table order; the
 *     segment of each non-empty one starts at the first multiple of the
 *     plan's segment alignment A at or after the end of the previous segment
 *     (0 for the first); an empty entry has no segment (its offset is the end
 *     so far rounded up to 16); payload_bytes = the end of the last segment
 *     rounded up to 16; every byte outside the segments is 0.  A = 16 by
 *     default: the segments follow each other at 16-byte alignment.  A
 *     larger A (fr_plan_create_ex; both sides of a transfer must use the
 *     same) leaves wider zero gaps: with A = 4096, tensors at scattered
 *     offsets pack and unpack faster, since every segment then starts on a
 *     4 KiB boundary.  Tables whose sent tensors are multiples of A bytes get
 *     the same payload for every A up to that size.
 *   Bitmaps.  Bit c of a result set lives in 32-bit word c / 32 at bit c % 32.
 *
 * Conventions
 *   All sizes and offsets are in bytes.  All device pointers are plain
 *   addresses of device memory on the plan's device; the caller owns every
 *   buffer.  The four operations validate synchronously, then enqueue on
 *   `stream` (a hipStream_t; NULL is the null stream) and return without
 *   waiting; their outputs are valid once the stream reaches that point.
 *   On any error nothing is enqueued and no output is touched.  A checksum or
 *   compare mismatch is data (a set bit and a count), not an error.
 *   Operations on one plan share the plan's device scratch: they must not run
 *   concurrently (issue them on one stream, or order the streams), and one
 *   plan must not be used from several host threads at once; use one plan per
 *   concurrent stream.
 *   Graph capture.  The four whole-state operations, fr_compare_sums and
 *   the flagged delta calls enqueue kernel launches only (no memset, no
 *   host copy, no allocation), so a capture of them into a HIP graph
 *   replays the same work.  The host-list delta calls copy the list from host memory: they
 *   are not for capture.
 */
#ifndef FLASHRESTORE_H
#define FLASHRESTORE_H

#include <stdint.h>

/* hipStream_t.  Like every HIP host header this needs the HIP platform
 * (hipcc defines it; a plain C or C++ compiler is given
 * -D__HIP_PLATFORM_AMD__ and the ROCm include directory). */
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#pragma GCC visibility push(default) /* the exported interface */
#endif

#define FR_ABI_VERSION 6

enum fr_dtype { FR_F32 = 1, FR_BF16 = 2 };

enum fr_status {
  FR_OK = 0,
  FR_E_INVAL = -1,           /* null required pointer, bad dtype, bad derive_from,
                                bad chunk_bytes, bad argument value */
  FR_E_ALIGN = -2,           /* an offset or a pointer not suitably aligned */
  FR_E_RANGE = -3,           /* an entry past its arena, a buffer too small or
                                past its allocation, too many chunks */
  FR_E_OVERLAP = -4,         /* overlapping receiver ranges or buffers */
  FR_E_NOMEM = -5,           /* host or device allocation failed */
  FR_E_DEVICE = -6,          /* a HIP call failed (see fr_last_hip_error) */
  FR_E_DEVICE_MISMATCH = -7  /* current device, stream or pointer not on the
                                plan's device */
};

/* One tensor of the state.  32 bytes, no padding. */
typedef struct fr_tensor_desc {
  uint64_t src_offset; /* from the sender / replica arena base; multiple of 16 */
  uint64_t dst_offset; /* from the receiver arena base; multiple of 16 */
  uint64_t numel;      /* elements; 0 allowed (no chunks, no payload) */
  uint32_t dtype;      /* FR_F32 or FR_BF16 */
  int32_t derive_from; /* -1, or the index of a non-derived FR_F32 entry with
                          the same numel; this entry must then be FR_BF16.  At
                          most one entry may derive from a given master. */
} fr_tensor_desc;

/* FRSUM-128 of one chunk.  16 bytes. */
typedef struct fr_chunk_sum {
  uint64_t sum;
  uint64_t wsum;
} fr_chunk_sum;

typedef struct fr_plan fr_plan; /* opaque, owned by the library */

typedef struct fr_plan_info {
  uint64_t n_entries;
  uint64_t chunk_bytes;
  uint64_t n_chunks;        /* total chunks; ids are < 2^32 */
  uint64_t payload_bytes;
  uint64_t bitmap_words;    /* ceil(n_chunks / 32) */
  uint64_t src_arena_bytes;
  uint64_t dst_arena_bytes;
  uint64_t state_bytes;     /* sum of nbytes over all entries */
  int64_t device;           /* HIP device the plan is bound to; -1 for a layout query */
  uint64_t segment_align;   /* A: payload segments start at multiples of it */
  uint64_t delta_payload_max; /* the largest delta payload any list of chunks can
                                 need: payload_bytes when chunk_bytes >= A, else
                                 the sent bytes plus A per sent chunk, rounded up
                                 to 16 */
  uint32_t pack_walk;       /* how fr_pack_state and fr_unpack_state divide their */
  uint32_t unpack_walk;     /* work (0 for a layout query): 0 slices of chunks,
                               1-3 slices cut at cache lines of one side, 4 one
                               aligned tile of the side written (the payload for
                               pack, the receiver arena for unpack) per workgroup,
                               the default where that side's chunks start inside
                               cache lines; FR_WALK_* */
  uint32_t tile_pack;       /* the tile each operation launches with, 0-10 (threads x */
  uint32_t tile_unpack;     /* 16-byte vectors per workgroup: 256x1, 512x1, 256x2, */
  uint32_t tile_verify;     /* 256x4, 64x4, 128x2, 64x2, 64x1, 128x1, 128x4, 64x8): */
  uint32_t tile_checksum;   /* set by FLASHRESTORE_TILE*, else chosen by chunk size;
                               a layout query reports what a plan created now, in
                               the same environment, would take */
} fr_plan_info;

#define FR_WALK_SLICES 0
#define FR_WALK_TILES 4

/* ---------------------------------------------------------------- plans */

/* Validate a tensor table and build a plan on the current HIP device.  The
 * table lists the model state a restore copies (Section II: parameters,
 * optimizer states and the rest of what training needs; Section III-E, its
 * part on restoring the model states); the plan fixes its chunks and payload
 * layout for every operation below.
 *   table            n_entries descriptors (host memory; copied)
 *   chunk_bytes      C: a power of two in [16, 2^30]
 *   src_arena_bytes  size of every sender / replica arena the plan will see
 *   dst_arena_bytes  size of every receiver arena
 *   out              receives the plan (unchanged on error)
 * Entries must lie inside their arenas (FR_E_RANGE), offsets must be
 * multiples of 16 (FR_E_ALIGN), receiver ranges must not overlap
 * (FR_E_OVERLAP; sender ranges may), the chunk count must be < 2^32
 * (FR_E_RANGE).  Synchronous: the plan's device tables are complete before
 * return.  They are copied and partly built by a kernel on a stream of the
 * call's own that does not synchronise with the null stream, and only that
 * stream is waited for, so work already queued elsewhere on the device is
 * neither waited for nor blocked.  Create plans outside graph capture, as
 * the allocations require.  The plan is immutable and bound to the device current at
 * creation.  Launch shapes are read from the environment at creation, and
 * results never depend on them: FLASHRESTORE_TILE (every operation) or
 * FLASHRESTORE_TILE_PACK / _UNPACK / _VERIFY / _CHECKSUM select a tile
 * 0-10 (threads x 16-byte vectors per workgroup: 256x1, 512x1, 256x2,
 * 256x4, 64x4, 128x2, 64x2, 64x1, 128x1, 128x4, 64x8; unset, by chunk
 * size: pack 64x4; unpack 64x1 up to 1 KiB chunks, 64x2 at 2 KiB, else
 * 128x2; compare 64x1 up to 2 KiB, else 128x2; checksum 64x4 up to 4 KiB,
 * 128x4 at 8 KiB, else 256x4), FLASHRESTORE_LINE (every
 * operation) or FLASHRESTORE_LINE_PACK / _UNPACK / _VERIFY / _CHECKSUM
 * choose how work is divided for data placed inside 128-byte lines: 0
 * plain slices of chunks, 1 slices cut at lines of the arena read (unpack:
 * of the receiver written), 2 (pack, unpack) at lines of the payload, 3
 * (pack, unpack) at slice boundaries of the payload, 4 (pack, unpack) one
 * aligned tile of the side written per workgroup (the payload for pack,
 * the receiver arena for unpack); unset, pack and unpack take 4 where the
 * side they write has chunks starting inside lines and 2 (pack) or 1
 * (unpack) otherwise, the compare 1 and the checksum 0 (fr_plan_info
 * reports the walks pack and unpack take and every operation's tile).  FLASHRESTORE_ABSORB_PACK / _UNPACK
 * / _VERIFY / _CHECKSUM (defaults 1, 1, 0, 0): a cut slice walk gives a
 * chunk's last slice its leftover lead instead of one more slice.
 * FLASHRESTORE_BUF_PACK / _UNPACK / _VERIFY / _CHECKSUM (default 0): slice
 * walks load through buffer resources, all of a thread's loads in flight
 * at once.  FLASHRESTORE_ORDER_VERIFY / _CHECKSUM (defaults 1, 0): the
 * compare's or the checksum's slices in arena address order rather than
 * chunk order (they differ for tables that list tensors out of arena
 * order).  FLASHRESTORE_MAX_GRID caps the workgroups per launch (0 or
 * unset: one per slice or tile). */
int fr_plan_create(const fr_tensor_desc* table, uint32_t n_entries, uint64_t chunk_bytes,
                   uint64_t src_arena_bytes, uint64_t dst_arena_bytes, fr_plan** out);

/* fr_plan_create with the payload segment alignment A given: a power of two
 * in [16, 2^20] (FR_E_INVAL otherwise).  fr_plan_create is A = 16.  The
 * payload (its size and every offset) depends on A, the sums and the
 * restored state do not. */
int fr_plan_create_ex(const fr_tensor_desc* table, uint32_t n_entries, uint64_t chunk_bytes,
                      uint64_t src_arena_bytes, uint64_t dst_arena_bytes, uint64_t segment_align,
                      fr_plan** out);

/* Sizes of a plan (the buffers a restore of Section III-E needs).  Host only. */
int fr_plan_get_info(const fr_plan* plan, fr_plan_info* out);

/* Global id of the chunk holding byte `byte_in_entry` of entry `entry`: the
 * chunk map that turns a flagged chunk back into (tensor, byte range), for a
 * restore check or replica compare (Sections III-A, III-E).  FR_E_RANGE if the
 * entry or byte does not exist.  Host only. */
int fr_plan_chunk_of(const fr_plan* plan, uint32_t entry, uint64_t byte_in_entry, uint64_t* chunk);

/* Payload offset of entry `entry` (UINT64_MAX for derived entries) and its
 * first chunk id: where a tensor's bytes travel in a restore (Section III-E),
 * e.g. to place stripes packed by several donors.  Host only. */
int fr_plan_entry_layout(const fr_plan* plan, uint32_t entry, uint64_t* payload_offset,
                         uint64_t* first_chunk, uint64_t* n_chunks);

/* Free a plan and its device tables (the end of the restore set-up of
 * fr_plan_create, Section III-E).  NULL is a no-op.  The caller must not
 * destroy a plan while work that uses it is still pending on a stream. */
int fr_plan_destroy(fr_plan* plan);

/* The same validation and layout as fr_plan_create_ex, on the host only,
 * with no device and no plan: fills `info` (device = -1) and, when non-NULL,
 * payload_offset[n_entries] (UINT64_MAX for derived entries) and
 * chunk_base[n_entries + 1]. */
int fr_layout_query(const fr_tensor_desc* table, uint32_t n_entries, uint64_t chunk_bytes,
                    uint64_t src_arena_bytes, uint64_t dst_arena_bytes, uint64_t segment_align,
                    fr_plan_info* info, uint64_t* payload_offset, uint64_t* chunk_base);

/* ----------------------------------------------------------- operations */

/* Donor side of a restore (Section III-E): payload <- the non-derived entries
 * of the arena at src_base, laid out as defined above with zero padding;
 * sums[c] <- FRSUM-128 of chunk c read from src_base, for every chunk,
 * derived entries included.
 *   src_base     device, 16-byte aligned, src_arena_bytes long
 *   payload      device, 16-byte aligned, payload_cap >= payload_bytes
 *   sums         device, 16-byte aligned, n_chunks entries
 * src, payload and sums must not overlap (FR_E_OVERLAP). */
int fr_pack_state(const fr_plan* plan, const void* src_base, void* payload, uint64_t payload_cap,
                  fr_chunk_sum* sums, hipStream_t stream);

/* Receiver side of a restore (Section III-E): for each non-derived entry copy
 * its payload segment to dst_base + dst_offset; for each derived entry write
 * RNE of the received master; then recompute FRSUM-128 of every chunk from
 * the bytes written and set bit c of bad_bitmap iff it differs from sums[c];
 * *n_bad = number of set bits.  Data is written even for bad chunks.  Bytes
 * of the receiver arena outside the entries are never written.
 *   payload      device, 16-byte aligned, payload_bytes long
 *   sums         device, 16-byte aligned, n_chunks entries (as sent)
 *   dst_base     device, 16-byte aligned, dst_arena_bytes long
 *   bad_bitmap   device, 4-byte aligned, bitmap_words words (may be NULL
 *                when n_chunks == 0); zeroed by the call
 *   n_bad        device, 8-byte aligned, one uint64; zeroed by the call
 * The receiver arena must not overlap any other argument. */
int fr_unpack_state(const fr_plan* plan, const void* payload, const fr_chunk_sum* sums,
                    void* dst_base, uint32_t* bad_bitmap, uint64_t* n_bad, hipStream_t stream);

/* Replica-consistency compare (Section III-A: data-parallel replicas must
 * hold the same state): bit c of diff_bitmap is set iff the bytes of chunk c
 * differ between the arenas at base_a and base_b (exact comparison, both
 * read at src offsets); *n_diff = number of set bits.  When sums_a / sums_b
 * are non-NULL they receive the chunk sums of each arena.  base_a == base_b
 * is allowed (empty result).  Outputs must not overlap inputs or each other. */
int fr_verify_replicas(const fr_plan* plan, const void* base_a, const void* base_b,
                       uint32_t* diff_bitmap, uint64_t* n_diff, fr_chunk_sum* sums_a,
                       fr_chunk_sum* sums_b, hipStream_t stream);

/* Replica-consistency check from chunk sums alone (Section III-A): for
 * replicas on different GPUs, each runs fr_checksum_state on its own arena
 * and the 16-byte sums travel instead of the state; bit c of diff_bitmap is
 * set iff sums_a[c] and sums_b[c] differ (either field); *n_diff = number of
 * set bits.  The bitmap drives fr_pack_flagged / fr_unpack_flagged like the
 * one fr_verify_replicas writes.  (Unlike that exact compare it sees only
 * what the sums see: every change of one or two bits of a chunk, see
 * FRSUM-128 above.)
 *   sums_a, sums_b  device, 16-byte aligned, n_chunks entries each
 *   diff_bitmap     device, 4-byte aligned, bitmap_words words; written
 *   n_diff          device, 8-byte aligned, one uint64; zeroed by the call
 * Outputs must not overlap the inputs or each other (FR_E_OVERLAP). */
int fr_compare_sums(const fr_plan* plan, const fr_chunk_sum* sums_a, const fr_chunk_sum* sums_b,
                    uint32_t* diff_bitmap, uint64_t* n_diff, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the replica
 * compare of fr_verify_replicas, with the same arguments, checks and outputs,
 * whose per-chunk flags and accumulators live in a static device array of
 * FR_STATIC_SCRATCH_BYTES that each GPU holds until the process ends, instead
 * of the plan's scratch.  The call allocates nothing (no hipMalloc, no
 * hipFree, no allocating library routine; the plan was built before).  Its
 * need is 4 * n_chunks bytes rounded up to 256, plus, when sums_a / sums_b
 * are requested, 32 * G * n_chunks bytes for G accumulators per chunk (G = 1
 * for chunks of up to 16 compare slices, C / (16 * slice bytes) above that);
 * a plan that needs more gets FR_E_RANGE with nothing enqueued.  Every such
 * call on one GPU shares that GPU's array, whatever its plan: calls that
 * overlap in time on one GPU (two streams, two threads) race and give wrong
 * results, so order them.  Each call clears what it uses first, so the
 * contents a previous call left do not matter. */
#define FR_STATIC_SCRATCH_BYTES (32ull << 20)
int fr_verify_replicas_noalloc(const fr_plan* plan, const void* base_a, const void* base_b,
                               uint32_t* diff_bitmap, uint64_t* n_diff, fr_chunk_sum* sums_a,
                               fr_chunk_sum* sums_b, hipStream_t stream);

/* Checksum of one replica's state (Section III-A: the replicas of a
 * data-parallel group hold the same state; Section III-E: a restore copies a
 * replica's state): sums[c] <- FRSUM-128 of chunk c of the arena at base
 * (src offsets); equal to the sums fr_pack_state produces for the same
 * bytes, so ranks can compare replicas, or check a restored state, by sums
 * alone. */
int fr_checksum_state(const fr_plan* plan, const void* base, fr_chunk_sum* sums, hipStream_t stream);

/* --------------------------------------------------------- delta repair */

/* Re-sending only the chunks in which a replica diverged, for example the set
 * fr_verify_replicas reports, instead of the whole state (the paper restores
 * from a data-parallel replica, Section III-E; a replica that differs from
 * its group in a few chunks needs only those).
 *   chunk_ids  host array of n_ids global chunk ids, strictly increasing,
 *              each < n_chunks (FR_E_INVAL otherwise); n_ids may be 0
 * Delta payload: the bytes of every listed chunk of a non-derived entry, in
 * list order; a chunk that directly follows the previous sent chunk of its
 * entry starts where that one ends, any other at the first multiple of the
 * plan's segment alignment A at or after it; the payload ends at the last
 * chunk's end rounded up to 16; every gap byte 0.  Listed chunks of derived
 * (bf16) entries send nothing.  With every chunk listed the delta payload and
 * sums equal fr_pack_state's; with C >= A the delta payload of a contiguous
 * range of chunk ids (a stripe) is fr_pack_state's payload from the range's
 * first sent chunk on, so stripes packed by several donors assemble into one
 * payload.
 * fr_delta_layout, fr_pack_chunks and fr_unpack_chunks take the list on the
 * host; fr_pack_flagged and fr_unpack_flagged take it as a device bitmap over
 * the chunk ids (bit c of word c / 32 set: chunk c listed; the list is the
 * set bits in increasing order), for example fr_verify_replicas's output, so
 * that a repair needs no host round trip.  Either way the device builds the
 * list's layout and unit records itself, in memory the plan allocated at
 * creation: no delta call allocates.  A host list is first copied to the
 * device on `stream` through pinned staging the plan owns (the call waits
 * until the previous copy from that staging has completed before refilling
 * it), so the host-list calls are not for graph capture; the flagged calls
 * enqueue kernel launches only and may be captured. */

/* Bytes of the delta payload for a list.  Host only.  (With C below A a
 * sparse list can need more than the full payload's payload_bytes, since
 * each chunk that does not continue the previous one starts on a multiple
 * of A.) */
int fr_delta_layout(const fr_plan* plan, const uint32_t* chunk_ids, uint64_t n_ids,
                    uint64_t* payload_bytes);

/* Donor side: payload <- the listed chunks as defined above; sums[i] <-
 * FRSUM-128 of chunk chunk_ids[i] read at src_base (derived chunks included).
 *   payload   device, 16-byte aligned, payload_cap >= fr_delta_layout bytes
 *   sums      device, 16-byte aligned, n_ids entries */
int fr_pack_chunks(const fr_plan* plan, const void* src_base, const uint32_t* chunk_ids,
                   uint64_t n_ids, void* payload, uint64_t payload_cap, fr_chunk_sum* sums,
                   hipStream_t stream);

/* Receiver side: write every sent chunk to dst_base; then recompute every
 * listed derived chunk as RNE of the receiver's master bytes (which by then
 * hold every sent master chunk); then set bit i of bad_bitmap iff FRSUM-128
 * of chunk chunk_ids[i] as written differs from sums[i]; *n_bad = number of
 * set bits.  Bytes outside the listed chunks are not written.
 *   payload        device, 16-byte aligned, as fr_pack_chunks wrote it for the
 *                  same list
 *   payload_bytes  bytes readable at payload; FR_E_RANGE if below the
 *                  fr_delta_layout bytes of the list
 *   sums           device, 16-byte aligned, n_ids entries
 *   bad_bitmap     device, 4-byte aligned, ceil(n_ids / 32) words (NULL if n_ids == 0)
 *   n_bad          device, 8-byte aligned, one uint64 */
int fr_unpack_chunks(const fr_plan* plan, const void* payload, uint64_t payload_bytes,
                     const fr_chunk_sum* sums, const uint32_t* chunk_ids, uint64_t n_ids,
                     void* dst_base, uint32_t* bad_bitmap, uint64_t* n_bad, hipStream_t stream);

/* Donor side of a repair from a device bitmap (the list is its set bits):
 * payload and sums as fr_pack_chunks for that list; sums[i] for list
 * position i < the list's length, rows past it untouched.
 *   flagged   device, 4-byte aligned, bitmap_words words (bits past n_chunks ignored)
 *   payload   device, 16-byte aligned, payload_cap >= delta_payload_max of the
 *             plan (fr_plan_get_info; FR_E_RANGE otherwise): the largest
 *             delta payload any list can need
 *   sums      device, 16-byte aligned, n_chunks entries
 *   counts    NULL, or device, 8-byte aligned, two uint64: the list's length
 *             and its delta payload bytes (what the transfer must carry) */
int fr_pack_flagged(const fr_plan* plan, const void* src_base, const uint32_t* flagged,
                    void* payload, uint64_t payload_cap, fr_chunk_sum* sums, uint64_t* counts,
                    hipStream_t stream);

/* Receiver side of a repair from a device bitmap: as fr_unpack_chunks for
 * the list of its set bits, with bits of bad_bitmap indexed by list
 * position; words past the list's end are written as 0.  A listed chunk
 * whose bytes lie past payload_bytes (the bytes readable at payload; pass
 * the donor's reported delta payload bytes or more) is neither read nor
 * written and its bit is set.
 *   payload     device, 16-byte aligned, payload_bytes long (0 allowed)
 *   sums        device, 16-byte aligned, n_chunks entries (as packed)
 *   flagged     device, 4-byte aligned, bitmap_words words: the same set as packed
 *   bad_bitmap  device, 4-byte aligned, bitmap_words words
 *   n_bad       device, 8-byte aligned, one uint64 */
int fr_unpack_flagged(const fr_plan* plan, const void* payload, uint64_t payload_bytes,
                      const fr_chunk_sum* sums, const uint32_t* flagged, void* dst_base,
                      uint32_t* bad_bitmap, uint64_t* n_bad, hipStream_t stream);

/* ------------------------------------------------- step tags and donors */

/* Host-only controller logic that decides *which* state a restore copies and
 * *when* the normal ranks may be stopped (Section III-E: its parts on the
 * step to resume from and on when to stop the normal processes).  Every rank tags
 * itself i when forward of step i starts, -1 when its optimizer step starts
 * and i+1 when that ends, and reports the tag with its heartbeat
 * (Section III-C).  A barrier merged into the gradient all-reduce keeps the
 * ranks in one phase, so once every normal rank reports the same tag T >= 0
 * the replicas hold the state at the start of step T: stop, restore the
 * failed ranks from replicas at step T, roll the data iterator back to T.
 * Readings where the paper is silent: a normal rank's tag counts only if it
 * was reported after the last failure was detected (an older report may show
 * i from a rank already inside its optimizer step); a rank silent for longer
 * than the timeout counts as failed, detected at last heartbeat + timeout;
 * fresh tags that are neither all equal nor -1 are inconsistent with the
 * barrier; a data-parallel group with no live rank leaves no replica, so the
 * answer is a checkpoint (Section III-G).  Times are seconds on any monotonic
 * clock; the timeout must exceed the heartbeat period. */

typedef struct fr_tracker fr_tracker; /* opaque, owned by the library */

enum fr_action {
  FR_ACT_CONTINUE = 0,            /* no failed rank */
  FR_ACT_WAIT = 1,                /* a normal rank is in its optimizer step or has not
                                     reported since the last failure was detected */
  FR_ACT_STOP_AND_RESTORE = 2,    /* stop, clean, reset; resume at resume_step */
  FR_ACT_CHECKPOINT_FALLBACK = 3, /* some data-parallel group has no live rank */
  FR_ACT_INCONSISTENT = 4         /* fresh normal tags disagree */
};

typedef struct fr_decision {
  int64_t resume_step; /* valid for FR_ACT_STOP_AND_RESTORE, else -1 */
  int32_t action;      /* enum fr_action */
  uint32_t n_failed;   /* ranks counted as failed */
  uint32_t n_waiting;  /* normal ranks the decision waits for */
  uint32_t reserved;
} fr_decision;

/* n_ranks > 0; dp_group[r] < n_ranks is the data-parallel group of rank r
 * (host array, copied; NULL puts every rank in group 0); timeout_s > 0. */
int fr_tracker_create(uint32_t n_ranks, const uint32_t* dp_group, double timeout_s, double now_s,
                      fr_tracker** out);
int fr_tracker_destroy(fr_tracker* t);
/* A heartbeat of `rank` carrying its tag (>= 0, or -1 in the optimizer step). */
int fr_tracker_heartbeat(fr_tracker* t, uint32_t rank, int64_t step_tag, double now_s);
/* A failure of `rank` reported by a monitor or device plugin at now_s. */
int fr_tracker_report_failure(fr_tracker* t, uint32_t rank, double now_s);
int fr_tracker_decide(const fr_tracker* t, double now_s, fr_decision* out);
/* The failed ranks in increasing order; FR_E_RANGE (with *n_failed set) if
 * more than cap. */
int fr_tracker_failed_ranks(const fr_tracker* t, double now_s, uint32_t* ranks, uint32_t cap,
                            uint32_t* n_failed);
/* donor[r] (n_ranks entries): for a failed rank, the live rank of its
 * data-parallel group whose state restores it (failed ranks of a group are
 * spread over its live ranks in rank order; Section III-D stage 3); -1 for
 * live ranks and for ranks whose group has no live rank. */
int fr_tracker_donors(const fr_tracker* t, double now_s, int32_t* donor);

/* ------------------------------------------ parallel layouts and donors */

/* Restore planning for data x tensor x pipeline parallel training with ZeRO
 * sharding (Section III-A lists DP, PP, TP and ZeRO/FSDP and their
 * combination; Section III-E restores vanilla DP, ZeRO/FSDP and combined
 * layouts from replicas).  Host only.  The paper fixes no rank order or shard
 * layout; this library's:
 *   world = tp * dp * pp; rank = t + tp * (d + dp * p) for tensor index t,
 *   data index d, pipeline index p.  The data-parallel group of a (t, p)
 *   slice is split into dp / shard replica groups of `shard` ranks:
 *   d = s + shard * q for shard index s and replica index q.
 *   zero_stage 0: vanilla DP (shard must be 1), every rank holds bf16
 *     params, fp32 master, m, v of every tensor of its slice;
 *   zero_stage 1 or 2: the slice's tensors are flattened in order into N
 *     elements, padded with zeros to a multiple of 8 * shard; shard s owns
 *     elements [s E, (s+1) E), E = N_pad / shard, of master, m and v; bf16
 *     params are kept whole;
 *   zero_stage 3: params are sharded like the optimizer state.
 * Ranks with equal (t, p, s) hold identical state and are each other's
 * replicas; a failed rank is restored from a live one of them. */
typedef struct fr_layout3d {
  uint32_t tp, pp, dp; /* parallel degrees, each >= 1 */
  uint32_t shard;      /* ranks a ZeRO shard group spans; divides dp */
  uint32_t zero_stage; /* 0, 1, 2 or 3 */
  uint32_t reserved;   /* 0 */
} fr_layout3d;

/* coords[5] <- (t, p, d, s, q) of `rank`. */
int fr_layout_rank_coords(const fr_layout3d* layout, uint32_t rank, uint32_t* coords);

/* failed[world] (0/1) -> donor[world]: for each failed rank a live replica
 * (failed ranks of a replica class are spread over its live ranks in rank
 * order), -1 for live ranks and for failed ranks with no live replica (those
 * need a checkpoint, Section III-G). */
int fr_layout_donors(const fr_layout3d* layout, const uint8_t* failed, int32_t* donor);

/* The tensor table of `rank`'s state arena (identical on all replicas of the
 * rank, so the donor packs and the new rank unpacks with the same plan):
 *   numel[n_tensors]  element counts of the slice's logical tensors
 * stage 0: per tensor [param bf16 (derived from the next), master, m, v];
 * stage 1/2: [param before the shard, param shard (derived from the master
 * shard), param after the shard, master shard, m shard, v shard];
 * stage 3: [param shard (derived), master shard, m shard, v shard].
 * Entries are contiguous, 16-aligned, src and dst offsets equal;
 * *arena_bytes = the arena size.  With table == NULL only *n_entries and
 * *arena_bytes are set; FR_E_RANGE if cap < *n_entries. */
int fr_layout_state_table(const fr_layout3d* layout, uint32_t rank, const uint64_t* numel,
                          uint32_t n_tensors, fr_tensor_desc* table, uint32_t cap,
                          uint32_t* n_entries, uint64_t* arena_bytes);

/* ---------------------------------------------------------------- misc */

const char* fr_strerror(int status);
int fr_last_hip_error(void); /* HIP error code behind the last FR_E_DEVICE on this thread */
int fr_abi_version(void);    /* FR_ABI_VERSION */

#if defined(__GNUC__)
#pragma GCC visibility pop
#endif

#ifdef __cplusplus
}
#endif
#endif /* FLASHRESTORE_H */
