/*
 * CPU oracle for data-parallel replica state restore.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark load this file's library.  The product
 * library never links, loads or calls it, and this file includes nothing of
 * the product's sources or headers.
 *
 * What is computed.  The paper restores the model state of a recreated
 * process from a healthy data-parallel replica by collective communication
 * instead of from a checkpoint (Section III-B item 3; Section III-E, its
 * part on restoring the model states), and the restored replica must be consistent
 * with the others again (Section III-A: data parallelism keeps model copies
 * consistent).  The paper fixes nothing below the level of copying the
 * replica's state; every format detail here is a reading, listed in the
 * design notes:
 *
 *   chunking   each tensor entry is cut into ceil(nbytes / C) byte chunks,
 *              only the last may be short; global chunk ids follow table
 *              order.
 *   FRSUM-128  a chunk's bytes read as little-endian 32-bit words w_i
 *              (missing tail bytes read as 0);  sum = sum_i w_i mod 2^64,
 *              wsum = sum_i (i+1) w_i mod 2^64.
 *   payload    the bytes of every non-derived entry in table order, each
 *              segment starting at the first multiple of the segment
 *              alignment `seg` (a power of two >= 16) at or after the end of
 *              the previous one (an empty entry has no segment), the payload
 *              ending at the last segment's end rounded up to 16, every gap
 *              byte 0.  seg = 16 packs the segments back to back; a larger
 *              seg (e.g. 4096) is the same rule with wider gaps.
 *              A bf16 entry that derives from an fp32 master is not sent;
 *              its chunk sums are.
 *   RNE        fp32 -> bf16: the nearer of the two neighbouring bf16 values,
 *              ties to an even last mantissa bit, overflow past the largest
 *              finite value to infinity, NaN -> (bits >> 16) | 0x0040.
 *   unpack     scatter the payload, re-derive bf16 = RNE(received master),
 *              recompute every chunk's FRSUM from the bytes written and flag
 *              each chunk whose sums differ from the sender's.
 *   verify     flag each chunk whose bytes differ between two replicas.
 *
 * It is written to be read, not to be fast: one pass per step, byte-level
 * definitions, OpenMP only across independent chunks.
 */
#include "fr_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static uint64_t esize_of(uint32_t dtype) { return dtype == ORO_F32 ? 4u : 2u; }
static uint64_t align16(uint64_t x) { return (x + 15u) & ~(uint64_t)15u; }
/* a payload segment starts at a multiple of seg (a power of two) */
static uint64_t align_segment(uint64_t x, uint64_t seg) { return (x + seg - 1) & ~(seg - 1); }
static int seg_ok(uint64_t seg) { return seg >= 16 && (seg & (seg - 1)) == 0; }

static int host_is_little_endian(void) {
  const uint32_t one = 1;
  unsigned char b;
  memcpy(&b, &one, 1);
  return b == 1;
}

/* ------------------------------------------------------------------ plan */

int oro_plan(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg, uint64_t* nchunks,
             uint64_t* chunk_base, uint64_t* pay_off, uint64_t* payload_bytes) {
  if (C == 0 || (C & (C - 1)) != 0 || !seg_ok(seg)) return -1;
  uint64_t base = 0, end = 0; /* end: where the last segment so far ends */
  for (uint32_t k = 0; k < n; k++) {
    uint64_t nb = t[k].numel * esize_of(t[k].dtype);
    uint64_t nc = (nb + C - 1) / C;
    nchunks[k] = nc;
    chunk_base[k] = base;
    base += nc;
    if (t[k].derive_from >= 0) {
      pay_off[k] = ORO_NO_PAYLOAD; /* derived entries are not sent */
    } else if (nb == 0) {
      pay_off[k] = align16(end); /* an empty entry occupies no segment */
    } else {
      pay_off[k] = align_segment(end, seg);
      end = pay_off[k] + nb;
    }
  }
  chunk_base[n] = base;
  *payload_bytes = align16(end);
  return 0;
}

/* ---------------------------------------------------------------- FRSUM-128 */

void oro_frsum(const uint8_t* p, uint64_t len, uint64_t* sum, uint64_t* wsum) {
  uint64_t s = 0, ws = 0;
  uint64_t nfull = len / 4;
  for (uint64_t i = 0; i < nfull; i++) {
    uint32_t w;
    memcpy(&w, p + 4 * i, 4); /* little-endian host: checked by oro_selfcheck */
    s += w;
    ws += (i + 1) * (uint64_t)w;
  }
  if (len % 4) { /* partial last word: present bytes in LE order, rest 0 */
    uint32_t w = 0;
    for (uint64_t b = 0; b < len % 4; b++) w |= (uint32_t)p[4 * nfull + b] << (8 * b);
    s += w;
    ws += (nfull + 1) * (uint64_t)w;
  }
  *sum = s;
  *wsum = ws;
}

/* -------------------------------------------------------------------- RNE */

/* Magnitude of a bf16 pattern as a double.  The pattern one past the largest
 * finite value (0x7F80, infinity) stands for 2^128 when rounding, as if the
 * exponent range were unbounded. */
static double bf16_magnitude(uint16_t h) {
  h &= 0x7FFF;
  if (h == 0x7F80) return ldexp(1.0, 128);
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

uint16_t oro_rne_bf16(uint32_t u) {
  uint32_t mag = u & 0x7FFFFFFFu;
  uint16_t sign = (uint16_t)((u >> 16) & 0x8000u);
  if (mag > 0x7F800000u) return (uint16_t)((u >> 16) | 0x0040u); /* NaN reading */
  if (mag == 0x7F800000u) return (uint16_t)(sign | 0x7F80u);      /* +-infinity */
  float f;
  memcpy(&f, &mag, 4);
  double x = (double)f;                 /* exact */
  uint16_t lo = (uint16_t)(mag >> 16);  /* largest bf16 magnitude <= x */
  if (bf16_magnitude(lo) == x) return (uint16_t)(sign | lo);
  uint16_t hi = (uint16_t)(lo + 1);     /* smallest bf16 magnitude > x */
  double dlo = x - bf16_magnitude(lo);  /* both differences are exact */
  double dhi = bf16_magnitude(hi) - x;
  uint16_t r;
  if (dlo < dhi) r = lo;
  else if (dhi < dlo) r = hi;
  else r = (lo & 1u) ? hi : lo; /* tie: the neighbour with an even last bit */
  return (uint16_t)(sign | r);
}

void oro_rne_bf16_array(const uint32_t* in, uint16_t* out, uint64_t n) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)n; i++) out[i] = oro_rne_bf16(in[i]);
}

/* ------------------------------------------------------------- operations */

static uint64_t chunk_len(uint64_t nbytes, uint64_t C, uint64_t j) {
  uint64_t start = j * C;
  uint64_t end = start + C < nbytes ? start + C : nbytes;
  return end - start;
}

/* Chunk sums of one arena at the entries' src offsets (or dst offsets). */
static void sums_of_arena(const oro_entry* t, uint32_t n, uint64_t C, const uint8_t* base,
                          int use_dst, const uint64_t* chunk_base, uint64_t* sums) {
  for (uint32_t k = 0; k < n; k++) {
    uint64_t nb = t[k].numel * esize_of(t[k].dtype);
    uint64_t nc = (nb + C - 1) / C;
    const uint8_t* e = base + (use_dst ? t[k].dst_offset : t[k].src_offset);
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t j = 0; j < (int64_t)nc; j++) {
      uint64_t c = chunk_base[k] + (uint64_t)j;
      oro_frsum(e + (uint64_t)j * C, chunk_len(nb, C, (uint64_t)j), &sums[2 * c], &sums[2 * c + 1]);
    }
  }
}

typedef struct {
  uint64_t* nchunks;
  uint64_t* chunk_base;
  uint64_t* pay_off;
  uint64_t payload_bytes;
} layout;

static int make_layout(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg, layout* L) {
  L->nchunks = (uint64_t*)malloc(sizeof(uint64_t) * (n + 1));
  L->chunk_base = (uint64_t*)malloc(sizeof(uint64_t) * (n + 1));
  L->pay_off = (uint64_t*)malloc(sizeof(uint64_t) * (n + 1));
  if (!L->nchunks || !L->chunk_base || !L->pay_off) return -1;
  return oro_plan(t, n, C, seg, L->nchunks, L->chunk_base, L->pay_off, &L->payload_bytes);
}

static void free_layout(layout* L) {
  free(L->nchunks);
  free(L->chunk_base);
  free(L->pay_off);
}

int oro_pack(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg, const uint8_t* src,
             uint8_t* payload, uint64_t* sums) {
  layout L;
  if (make_layout(t, n, C, seg, &L)) return -1;
  memset(payload, 0, L.payload_bytes);
  for (uint32_t k = 0; k < n; k++) {
    if (t[k].derive_from >= 0) continue;
    memcpy(payload + L.pay_off[k], src + t[k].src_offset, t[k].numel * esize_of(t[k].dtype));
  }
  sums_of_arena(t, n, C, src, 0, L.chunk_base, sums);
  free_layout(&L);
  return 0;
}

int oro_unpack(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg, const uint8_t* payload,
               const uint64_t* sums, uint8_t* dst, uint32_t* bitmap, uint64_t* n_bad) {
  layout L;
  if (make_layout(t, n, C, seg, &L)) return -1;
  uint64_t total = L.chunk_base[n];
  for (uint32_t k = 0; k < n; k++) {
    if (t[k].derive_from >= 0) continue;
    memcpy(dst + t[k].dst_offset, payload + L.pay_off[k], t[k].numel * esize_of(t[k].dtype));
  }
  for (uint32_t k = 0; k < n; k++) {
    int32_t s = t[k].derive_from;
    if (s < 0) continue;
    const uint8_t* master = payload + L.pay_off[s];
    uint8_t* out = dst + t[k].dst_offset;
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < (int64_t)t[k].numel; e++) {
      uint32_t u;
      memcpy(&u, master + 4 * (uint64_t)e, 4);
      uint16_t h = oro_rne_bf16(u);
      memcpy(out + 2 * (uint64_t)e, &h, 2);
    }
  }
  uint64_t* got = (uint64_t*)malloc(sizeof(uint64_t) * 2 * (total ? total : 1));
  if (!got) return -1;
  sums_of_arena(t, n, C, dst, 1, L.chunk_base, got);
  memset(bitmap, 0, sizeof(uint32_t) * ((total + 31) / 32));
  uint64_t bad = 0;
  for (uint64_t c = 0; c < total; c++) {
    if (got[2 * c] != sums[2 * c] || got[2 * c + 1] != sums[2 * c + 1]) {
      bitmap[c / 32] |= 1u << (c % 32);
      bad++;
    }
  }
  *n_bad = bad;
  free(got);
  free_layout(&L);
  return 0;
}

int oro_verify(const oro_entry* t, uint32_t n, uint64_t C, const uint8_t* a, const uint8_t* b,
               uint32_t* bitmap, uint64_t* n_diff, uint64_t* sums_a, uint64_t* sums_b) {
  layout L;
  if (make_layout(t, n, C, 16, &L)) return -1;  /* chunk map only */
  uint64_t total = L.chunk_base[n];
  uint8_t* differs = (uint8_t*)calloc(total ? total : 1, 1);
  if (!differs) return -1;
  for (uint32_t k = 0; k < n; k++) {
    uint64_t nb = t[k].numel * esize_of(t[k].dtype);
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t j = 0; j < (int64_t)L.nchunks[k]; j++) {
      uint64_t off = t[k].src_offset + (uint64_t)j * C;
      differs[L.chunk_base[k] + (uint64_t)j] =
          memcmp(a + off, b + off, chunk_len(nb, C, (uint64_t)j)) != 0;
    }
  }
  memset(bitmap, 0, sizeof(uint32_t) * ((total + 31) / 32));
  uint64_t cnt = 0;
  for (uint64_t c = 0; c < total; c++) {
    if (differs[c]) {
      bitmap[c / 32] |= 1u << (c % 32);
      cnt++;
    }
  }
  *n_diff = cnt;
  if (sums_a) sums_of_arena(t, n, C, a, 0, L.chunk_base, sums_a);
  if (sums_b) sums_of_arena(t, n, C, b, 0, L.chunk_base, sums_b);
  free(differs);
  free_layout(&L);
  return 0;
}

int oro_checksum(const oro_entry* t, uint32_t n, uint64_t C, const uint8_t* base, uint64_t* sums) {
  layout L;
  if (make_layout(t, n, C, 16, &L)) return -1;  /* chunk map only */
  sums_of_arena(t, n, C, base, 0, L.chunk_base, sums);
  free_layout(&L);
  return 0;
}

/* Chunk sums of an explicit list of chunks: the sampled form used on
 * workloads too large to run whole.  chunk ids are global ids. */
int oro_checksum_chunks(const oro_entry* t, uint32_t n, uint64_t C, const uint8_t* base,
                        const uint64_t* ids, uint64_t n_ids, uint64_t* sums) {
  layout L;
  if (make_layout(t, n, C, 16, &L)) return -1;  /* chunk map only */
  for (uint64_t q = 0; q < n_ids; q++) {
    uint64_t c = ids[q];
    uint32_t lo = 0, hi = n; /* entry k with chunk_base[k] <= c < chunk_base[k+1] */
    while (hi - lo > 1) {
      uint32_t mid = lo + (hi - lo) / 2;
      if (L.chunk_base[mid] <= c) lo = mid; else hi = mid;
    }
    uint64_t j = c - L.chunk_base[lo];
    uint64_t nb = t[lo].numel * esize_of(t[lo].dtype);
    oro_frsum(base + t[lo].src_offset + j * C, chunk_len(nb, C, j), &sums[2 * q], &sums[2 * q + 1]);
  }
  free_layout(&L);
  return 0;
}

/* Replica-consistency check from sums alone (Section III-A): a chunk is
 * flagged when either of its two sums differs between the replicas. */
int oro_compare_sums(const uint64_t* a, const uint64_t* b, uint64_t n_chunks, uint32_t* bitmap,
                     uint64_t* n_diff) {
  uint64_t nd = 0;
  for (uint64_t w = 0; w < (n_chunks + 31) / 32; w++) bitmap[w] = 0;
  for (uint64_t c = 0; c < n_chunks; c++) {
    if (a[2 * c] != b[2 * c] || a[2 * c + 1] != b[2 * c + 1]) {
      bitmap[c / 32] |= 1u << (c % 32);
      nd++;
    }
  }
  *n_diff = nd;
  return 0;
}

/* ------------------------------------------------------------ delta repair
 *
 * Re-sending only the chunks in which a replica diverged.  The caller lists
 * global chunk ids in strictly increasing order.  Delta payload: the bytes of
 * every listed chunk of a non-derived entry, in list order; a chunk that
 * directly follows the previous sent chunk in its entry starts where that one
 * ends, any other at the next multiple of the segment alignment; the payload ends
 * at the last chunk's end rounded up to 16; every gap byte 0.  (With every
 * chunk listed this is the full payload.)  Listed chunks of a derived (bf16)
 * entry send nothing.  sums[i] is the FRSUM of chunk ids[i] at the sender.
 * At the receiver the sent chunks are written first; then each listed derived
 * chunk is recomputed as RNE of the receiver's master bytes (which now hold
 * every sent master chunk); then every listed chunk is checked, bit i of the
 * result standing for list position i. */

typedef struct {
  uint32_t entry;
  uint64_t j; /* chunk index within the entry */
} chunk_loc;

static chunk_loc locate(const layout* L, uint32_t n, uint64_t c) {
  uint32_t lo = 0, hi = n; /* entry k with chunk_base[k] <= c < chunk_base[k+1] */
  while (hi - lo > 1) {
    uint32_t mid = lo + (hi - lo) / 2;
    if (L->chunk_base[mid] <= c) lo = mid; else hi = mid;
  }
  chunk_loc r = {lo, c - L->chunk_base[lo]};
  return r;
}

static int list_ok(const layout* L, uint32_t n, const uint32_t* ids, uint64_t n_ids) {
  for (uint64_t i = 0; i < n_ids; i++) {
    if (ids[i] >= L->chunk_base[n]) return 0;
    if (i && ids[i] <= ids[i - 1]) return 0;
  }
  return 1;
}

int oro_delta_layout(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg, const uint32_t* ids,
                     uint64_t n_ids, uint64_t* pay_off, uint64_t* payload_bytes) {
  layout L;
  if (make_layout(t, n, C, seg, &L)) return -1;
  if (!list_ok(&L, n, ids, n_ids)) { free_layout(&L); return -1; }
  uint64_t end = 0;
  int have_prev = 0;
  chunk_loc prev = {0, 0};
  for (uint64_t i = 0; i < n_ids; i++) {
    chunk_loc w = locate(&L, n, ids[i]);
    if (t[w.entry].derive_from >= 0) {
      pay_off[i] = ORO_NO_PAYLOAD;
    } else {
      uint64_t nb = t[w.entry].numel * esize_of(t[w.entry].dtype);
      int follows = have_prev && prev.entry == w.entry && prev.j + 1 == w.j;
      pay_off[i] = follows ? end : align_segment(end, seg);
      end = pay_off[i] + chunk_len(nb, C, w.j);
      prev = w;
      have_prev = 1;
    }
  }
  *payload_bytes = align16(end);
  free_layout(&L);
  return 0;
}

int oro_pack_chunks(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg, const uint8_t* src,
                    const uint32_t* ids, uint64_t n_ids, uint8_t* payload, uint64_t* sums) {
  uint64_t* off = (uint64_t*)malloc(sizeof(uint64_t) * (n_ids ? n_ids : 1));
  uint64_t pb;
  if (!off || oro_delta_layout(t, n, C, seg, ids, n_ids, off, &pb)) { free(off); return -1; }
  layout L;
  if (make_layout(t, n, C, seg, &L)) { free(off); return -1; }
  memset(payload, 0, pb);
  for (uint64_t i = 0; i < n_ids; i++) {
    chunk_loc w = locate(&L, n, ids[i]);
    uint64_t nb = t[w.entry].numel * esize_of(t[w.entry].dtype);
    uint64_t len = chunk_len(nb, C, w.j);
    const uint8_t* from = src + t[w.entry].src_offset + w.j * C;
    if (off[i] != ORO_NO_PAYLOAD) memcpy(payload + off[i], from, len);
    oro_frsum(from, len, &sums[2 * i], &sums[2 * i + 1]);
  }
  free_layout(&L);
  free(off);
  return 0;
}

int oro_unpack_chunks(const oro_entry* t, uint32_t n, uint64_t C, uint64_t seg,
                      const uint8_t* payload,
                      const uint64_t* sums, const uint32_t* ids, uint64_t n_ids, uint8_t* dst,
                      uint32_t* bitmap, uint64_t* n_bad) {
  uint64_t* off = (uint64_t*)malloc(sizeof(uint64_t) * (n_ids ? n_ids : 1));
  uint64_t pb;
  if (!off || oro_delta_layout(t, n, C, seg, ids, n_ids, off, &pb)) { free(off); return -1; }
  layout L;
  if (make_layout(t, n, C, seg, &L)) { free(off); return -1; }
  /* 1. the sent chunks */
  for (uint64_t i = 0; i < n_ids; i++) {
    if (off[i] == ORO_NO_PAYLOAD) continue;
    chunk_loc w = locate(&L, n, ids[i]);
    uint64_t nb = t[w.entry].numel * esize_of(t[w.entry].dtype);
    memcpy(dst + t[w.entry].dst_offset + w.j * C, payload + off[i], chunk_len(nb, C, w.j));
  }
  /* 2. derived chunks from the receiver's masters */
  for (uint64_t i = 0; i < n_ids; i++) {
    if (off[i] != ORO_NO_PAYLOAD) continue;
    chunk_loc w = locate(&L, n, ids[i]);
    const oro_entry* e = &t[w.entry];
    const oro_entry* m = &t[e->derive_from];
    uint64_t len = chunk_len(e->numel * 2, C, w.j);
    uint64_t first = w.j * C / 2; /* first element of the chunk */
    for (uint64_t q = 0; q < len / 2; q++) {
      uint32_t u;
      memcpy(&u, dst + m->dst_offset + 4 * (first + q), 4);
      uint16_t h = oro_rne_bf16(u);
      memcpy(dst + e->dst_offset + 2 * (first + q), &h, 2);
    }
  }
  /* 3. check every listed chunk as written */
  memset(bitmap, 0, sizeof(uint32_t) * ((n_ids + 31) / 32));
  uint64_t bad = 0;
  for (uint64_t i = 0; i < n_ids; i++) {
    chunk_loc w = locate(&L, n, ids[i]);
    uint64_t nb = t[w.entry].numel * esize_of(t[w.entry].dtype);
    uint64_t s, ws;
    oro_frsum(dst + t[w.entry].dst_offset + w.j * C, chunk_len(nb, C, w.j), &s, &ws);
    if (s != sums[2 * i] || ws != sums[2 * i + 1]) {
      bitmap[i / 32] |= 1u << (i % 32);
      bad++;
    }
  }
  *n_bad = bad;
  free_layout(&L);
  free(off);
  return 0;
}

int oro_selfcheck(void) { return host_is_little_endian() ? 0 : -1; }

int oro_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads for the following calls (timing only; results never depend on it). */
void oro_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}
