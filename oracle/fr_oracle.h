/*
 * CPU oracle for data-parallel replica state restore: declarations.
 * TEST INFRASTRUCTURE ONLY (see fr_oracle.c).  Independent of the product
 * library's headers; the descriptor layout is the same 32-byte input format
 * because both sides read the same tables.
 */
#ifndef FR_ORACLE_H
#define FR_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORO_F32 = 1, ORO_BF16 = 2 };
#define ORO_NO_PAYLOAD UINT64_MAX
/* Payload layout (a reading: the paper fixes no wire format): the sent
 * entries' bytes in table order, each non-empty one starting at the first
 * multiple of the segment alignment `seg` at or after the end of the previous
 * one, the whole payload ending at the last entry's end rounded up to 16;
 * every other byte 0.  An empty entry's offset is the end so far rounded up
 * to 16.  seg is a power of two >= 16: 16 packs the entries back to back
 * (the default reading), larger values leave wider zero gaps. */

typedef struct {
  uint64_t src_offset; /* byte offset in the sender / replica arena */
  uint64_t dst_offset; /* byte offset in the receiver arena */
  uint64_t numel;
  uint32_t dtype;      /* ORO_F32 or ORO_BF16 */
  int32_t derive_from; /* -1, or index of the fp32 master of a bf16 entry */
} oro_entry;

/* Layout: per-entry chunk counts, chunk bases (n+1 values, last = total) and
 * payload offsets (ORO_NO_PAYLOAD for derived entries). */
int oro_plan(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg, uint64_t* nchunks,
             uint64_t* chunk_base, uint64_t* pay_off, uint64_t* payload_bytes);

/* FRSUM-128 of len bytes. */
void oro_frsum(const uint8_t* p, uint64_t len, uint64_t* sum, uint64_t* wsum);

/* fp32 bit pattern -> bf16 bit pattern, round to nearest even. */
uint16_t oro_rne_bf16(uint32_t u);
void oro_rne_bf16_array(const uint32_t* in, uint16_t* out, uint64_t n);

/* sums arrays hold 2 x u64 (sum, wsum) per chunk. */
int oro_pack(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg, const uint8_t* src,
             uint8_t* payload, uint64_t* sums);
int oro_unpack(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg, const uint8_t* payload,
               const uint64_t* sums, uint8_t* dst, uint32_t* bitmap, uint64_t* n_bad);
int oro_verify(const oro_entry* t, uint32_t n, uint64_t C, const uint8_t* a, const uint8_t* b,
               uint32_t* bitmap, uint64_t* n_diff, uint64_t* sums_a, uint64_t* sums_b);
int oro_checksum(const oro_entry* t, uint32_t n, uint64_t C, const uint8_t* base, uint64_t* sums);
int oro_checksum_chunks(const oro_entry* t, uint32_t n, uint64_t C, const uint8_t* base,
                        const uint64_t* ids, uint64_t n_ids, uint64_t* sums);
/* Replica-consistency check from sums alone (Section III-A): bit c of
 * bitmap set iff chunk c's (sum, wsum) differ between a and b (2 words per
 * chunk each); *n_diff = set bits.  bitmap: ceil(n_chunks / 32) words. */
int oro_compare_sums(const uint64_t* a, const uint64_t* b, uint64_t n_chunks, uint32_t* bitmap,
                     uint64_t* n_diff);

/* Delta repair over a strictly increasing list of global chunk ids (see
 * fr_oracle.c).  pay_off[i] is ORO_NO_PAYLOAD for derived chunks; bitmap and
 * sums are indexed by list position. */
int oro_delta_layout(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg, const uint32_t* ids,
                     uint64_t n_ids, uint64_t* pay_off, uint64_t* payload_bytes);
int oro_pack_chunks(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg, const uint8_t* src,
                    const uint32_t* ids, uint64_t n_ids, uint8_t* payload, uint64_t* sums);
int oro_unpack_chunks(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg,
                      const uint8_t* payload,
                      const uint64_t* sums, const uint32_t* ids, uint64_t n_ids, uint8_t* dst,
                      uint32_t* bitmap, uint64_t* n_bad);

int oro_selfcheck(void);
int oro_threads(void);
void oro_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
