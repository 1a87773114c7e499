/*
 * A plain C program that drives libflashrestore through its C ABI with raw
 * HIP device memory and a HIP stream (no Python, no torch): restore a small
 * state across differing sender and receiver layouts, compare two replicas,
 * checksum, repair the diverged replica by a delta, and check every output
 * byte against the C oracle.  Test
 * infrastructure: built by the package build, run by
 * tests/test_gpu_c_abi.py.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "flashrestore.h"
#include "fr_oracle.h"

#define HIP(x)                                                                  \
  do {                                                                          \
    hipError_t e_ = (x);                                                        \
    if (e_ != hipSuccess) {                                                     \
      fprintf(stderr, "HIP error %d: %s (line %d)\n", (int)e_, #x, __LINE__);   \
      return 1;                                                                 \
    }                                                                           \
  } while (0)
#define FR(x)                                                                   \
  do {                                                                          \
    int rc_ = (x);                                                              \
    if (rc_ != FR_OK) {                                                         \
      fprintf(stderr, "%s -> %d (%s), line %d\n", #x, rc_, fr_strerror(rc_), __LINE__); \
      return 1;                                                                 \
    }                                                                           \
  } while (0)
#define CHECK(c, msg)                                            \
  do {                                                           \
    if (!(c)) {                                                  \
      fprintf(stderr, "FAILED: %s (line %d)\n", msg, __LINE__);  \
      return 1;                                                  \
    }                                                            \
  } while (0)

enum { N_TENSORS = 4, N_ENTRIES = 4 * N_TENSORS };

static uint64_t mix(uint64_t x) { /* splitmix64 finaliser */
  x += 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  return x ^ (x >> 31);
}

static uint64_t up16(uint64_t x) { return (x + 15) & ~(uint64_t)15; }

int main(void) {
  /* four logical tensors: bf16 parameter derived from its fp32 master, the
   * master, Adam m and v; odd sizes make ragged chunk tails */
  const uint64_t numel[N_TENSORS] = {1000003, 4096, 77, 65537};
  const uint64_t C = 16384;
  fr_tensor_desc t[N_ENTRIES];
  oro_entry o[N_ENTRIES];
  uint64_t so = 0, dof = 0;
  for (int k = 0; k < N_TENSORS; k++) {
    for (int a = 0; a < 4; a++) {
      const int e = 4 * k + a;
      const uint64_t nb = numel[k] * (a == 0 ? 2 : 4);
      t[e].src_offset = so;
      t[e].dst_offset = dof + 16 * (uint64_t)(e % 3); /* receiver gaps differ */
      t[e].numel = numel[k];
      t[e].dtype = a == 0 ? FR_BF16 : FR_F32;
      t[e].derive_from = a == 0 ? e + 1 : -1;
      so += up16(nb);
      dof = t[e].dst_offset + up16(nb);
      o[e].src_offset = t[e].src_offset;
      o[e].dst_offset = t[e].dst_offset;
      o[e].numel = t[e].numel;
      o[e].dtype = t[e].dtype;
      o[e].derive_from = t[e].derive_from;
    }
  }
  const uint64_t src_bytes = so, dst_bytes = dof;

  /* sender state: master and moments from a counter-based generator, the
   * parameter rounded from the master */
  uint8_t* src = calloc(src_bytes, 1);
  CHECK(src, "host allocation");
  for (int e = 0; e < N_ENTRIES; e++) {
    if (t[e].dtype != FR_F32) continue;
    uint32_t* w = (uint32_t*)(src + t[e].src_offset);
    for (uint64_t i = 0; i < t[e].numel; i++) {
      const uint64_t r = mix(((uint64_t)e << 40) ^ i);
      float f = (float)((int32_t)(uint32_t)r) * 1e-11f; /* about +-0.02 */
      memcpy(&w[i], &f, 4);
    }
  }
  for (int e = 0; e < N_ENTRIES; e++) {
    if (t[e].derive_from < 0) continue;
    const uint32_t* m = (const uint32_t*)(src + t[t[e].derive_from].src_offset);
    uint16_t* p = (uint16_t*)(src + t[e].src_offset);
    oro_rne_bf16_array(m, p, t[e].numel);
  }

  /* the oracle's outputs */
  uint64_t nch[N_ENTRIES], base[N_ENTRIES + 1], pay[N_ENTRIES], pb = 0;
  CHECK(oro_plan(o, N_ENTRIES, C, 16, nch, base, pay, &pb) == 0, "oracle plan");
  const uint64_t n = base[N_ENTRIES];
  uint8_t* o_pay = calloc(pb ? pb : 1, 1);
  uint64_t* o_sums = calloc(2 * n, 8);
  uint8_t* o_dst = malloc(dst_bytes);
  uint32_t* o_bm = calloc((n + 31) / 32, 4);
  uint64_t o_nbad = 0;
  CHECK(o_pay && o_sums && o_dst && o_bm, "host allocation");
  memset(o_dst, 0x5A, dst_bytes);
  CHECK(oro_pack(o, N_ENTRIES, C, 16, src, o_pay, o_sums) == 0, "oracle pack");
  CHECK(oro_unpack(o, N_ENTRIES, C, 16, o_pay, o_sums, o_dst, o_bm, &o_nbad) == 0 && o_nbad == 0,
        "oracle unpack");

  /* device buffers and a stream of default priority */
  hipStream_t s;
  HIP(hipStreamCreate(&s));
  void *d_src, *d_dst, *d_pay, *d_rep;
  fr_chunk_sum *d_sums, *d_csum;
  uint32_t *d_bm, *d_diff;
  uint64_t *d_nbad, *d_ndiff;
  const uint64_t words = (n + 31) / 32;
  HIP(hipMalloc(&d_src, src_bytes));
  HIP(hipMalloc(&d_rep, src_bytes));
  HIP(hipMalloc(&d_dst, dst_bytes));
  HIP(hipMalloc(&d_pay, pb));
  HIP(hipMalloc((void**)&d_sums, n * sizeof(fr_chunk_sum)));
  HIP(hipMalloc((void**)&d_csum, n * sizeof(fr_chunk_sum)));
  HIP(hipMalloc((void**)&d_bm, words * 4));
  HIP(hipMalloc((void**)&d_diff, words * 4));
  HIP(hipMalloc((void**)&d_nbad, 8));
  HIP(hipMalloc((void**)&d_ndiff, 8));
  HIP(hipMemcpy(d_src, src, src_bytes, hipMemcpyHostToDevice));
  HIP(hipMemset(d_dst, 0x5A, dst_bytes));
  HIP(hipMemset(d_pay, 0xEE, pb)); /* pack must write padding and gaps */

  fr_plan* plan = NULL;
  FR(fr_plan_create(t, N_ENTRIES, C, src_bytes, dst_bytes, &plan));
  fr_plan_info info;
  FR(fr_plan_get_info(plan, &info));
  CHECK(info.n_chunks == n && info.payload_bytes == pb, "plan sizes equal the oracle's");

  /* errors return their code and enqueue nothing */
  CHECK(fr_pack_state(plan, d_src, d_pay, pb - 1, d_sums, s) == FR_E_RANGE, "payload too small");
  CHECK(fr_pack_state(plan, (uint8_t*)d_src + 8, d_pay, pb, d_sums, s) == FR_E_ALIGN, "misaligned");
  CHECK(fr_unpack_state(plan, d_pay, d_sums, d_dst, d_bm, NULL, s) == FR_E_INVAL, "null counter");

  /* restore: pack on the donor, unpack on the receiver */
  FR(fr_pack_state(plan, d_src, d_pay, pb, d_sums, s));
  FR(fr_unpack_state(plan, d_pay, d_sums, d_dst, d_bm, d_nbad, s));
  FR(fr_checksum_state(plan, d_src, d_csum, s));
  HIP(hipStreamSynchronize(s));
  uint8_t* g_pay = malloc(pb);
  uint64_t* g_sums = malloc(n * 16);
  uint64_t* g_csum = malloc(n * 16);
  uint8_t* g_dst = malloc(dst_bytes);
  uint32_t* g_bm = malloc(words * 4);
  uint64_t g_nbad = 99, g_ndiff = 99;
  CHECK(g_pay && g_sums && g_csum && g_dst && g_bm, "host allocation");
  HIP(hipMemcpy(g_pay, d_pay, pb, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(g_sums, d_sums, n * 16, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(g_csum, d_csum, n * 16, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(g_dst, d_dst, dst_bytes, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(g_bm, d_bm, words * 4, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(&g_nbad, d_nbad, 8, hipMemcpyDeviceToHost));
  CHECK(memcmp(g_pay, o_pay, pb) == 0, "payload equals the oracle's");
  CHECK(memcmp(g_sums, o_sums, n * 16) == 0, "sums equal the oracle's");
  CHECK(memcmp(g_csum, o_sums, n * 16) == 0, "checksum equals the pack sums");
  CHECK(memcmp(g_dst, o_dst, dst_bytes) == 0, "receiver arena equals the oracle's");
  CHECK(g_nbad == 0 && memcmp(g_bm, o_bm, words * 4) == 0, "nothing flagged");

  /* replica compare: one flipped bit is located to its chunk */
  const uint32_t entry = 9;                 /* tensor 2's master */
  const uint64_t byte_in_entry = 101;
  uint64_t chunk = 0;
  FR(fr_plan_chunk_of(plan, entry, byte_in_entry, &chunk));
  HIP(hipMemcpy(d_rep, d_src, src_bytes, hipMemcpyDeviceToDevice));
  uint8_t b = 0;
  uint8_t* at = (uint8_t*)d_rep + t[entry].src_offset + byte_in_entry;
  HIP(hipMemcpy(&b, at, 1, hipMemcpyDeviceToHost));
  b ^= 0x10;
  HIP(hipMemcpy(at, &b, 1, hipMemcpyHostToDevice));
  FR(fr_verify_replicas(plan, d_src, d_rep, d_diff, d_ndiff, NULL, NULL, s));
  HIP(hipStreamSynchronize(s));
  HIP(hipMemcpy(g_bm, d_diff, words * 4, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(&g_ndiff, d_ndiff, 8, hipMemcpyDeviceToHost));
  CHECK(g_ndiff == 1, "one chunk differs");
  for (uint64_t c = 0; c < n; c++)
    CHECK(((g_bm[c / 32] >> (c % 32)) & 1u) == (c == chunk), "the flipped chunk is flagged");

  /* delta repair: re-send the flagged chunk and a derived parameter chunk
   * (recomputed from the receiver's master) into the diverged replica.
   * Replicas share the donor's layout, so the repair plan's receiver layout
   * is the sender's (chunk ids are the same in both plans).  This plan
   * places payload segments on 4 KiB boundaries, the main one packs them. */
  fr_tensor_desc t2[N_ENTRIES];
  oro_entry o2[N_ENTRIES];
  memcpy(t2, t, sizeof t);
  memcpy(o2, o, sizeof o);
  for (int e = 0; e < N_ENTRIES; e++) t2[e].dst_offset = o2[e].dst_offset = t[e].src_offset;
  fr_plan* rplan = NULL;
  FR(fr_plan_create_ex(t2, N_ENTRIES, C, src_bytes, src_bytes, 4096, &rplan));
  const uint32_t ids[2] = {0u, (uint32_t)chunk};
  uint64_t dpb = 0, o_dpb = 0, o_doff[2];
  FR(fr_delta_layout(rplan, ids, 2, &dpb));
  CHECK(oro_delta_layout(o2, N_ENTRIES, C, 4096, ids, 2, o_doff, &o_dpb) == 0 && dpb == o_dpb,
        "delta payload size equals the oracle's");
  uint8_t* o_dpay = calloc(dpb, 1);
  uint64_t o_dsums[4];
  CHECK(o_dpay && oro_pack_chunks(o2, N_ENTRIES, C, 4096, src, ids, 2, o_dpay, o_dsums) == 0,
        "oracle delta pack");
  void* d_dpay;
  fr_chunk_sum* d_dsums;
  uint32_t* d_dbm;
  HIP(hipMalloc(&d_dpay, dpb));
  HIP(hipMalloc((void**)&d_dsums, 2 * sizeof(fr_chunk_sum)));
  HIP(hipMalloc((void**)&d_dbm, 4));
  CHECK(fr_unpack_chunks(plan, d_dpay, dpb, d_dsums, ids, 2, d_rep, d_dbm, d_nbad, s) ==
            FR_E_RANGE, "a replica arena smaller than the plan's receiver arena");
  CHECK(fr_unpack_chunks(rplan, d_dpay, dpb - 16, d_dsums, ids, 2, d_rep, d_dbm, d_nbad, s) ==
            FR_E_RANGE, "delta payload shorter than the list needs");
  FR(fr_pack_chunks(rplan, d_src, ids, 2, d_dpay, dpb, d_dsums, s));
  FR(fr_unpack_chunks(rplan, d_dpay, dpb, d_dsums, ids, 2, d_rep, d_dbm, d_nbad, s));
  HIP(hipStreamSynchronize(s));
  uint8_t* g_dpay = malloc(dpb);
  uint64_t g_dsums[4];
  uint8_t* g_rep = malloc(src_bytes);
  CHECK(g_dpay && g_rep, "host allocation");
  HIP(hipMemcpy(g_dpay, d_dpay, dpb, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(g_dsums, d_dsums, 32, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(g_rep, d_rep, src_bytes, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(&g_nbad, d_nbad, 8, hipMemcpyDeviceToHost));
  CHECK(memcmp(g_dpay, o_dpay, dpb) == 0 && memcmp(g_dsums, o_dsums, 32) == 0,
        "delta payload and sums equal the oracle's");
  CHECK(g_nbad == 0 && memcmp(g_rep, src, src_bytes) == 0, "the replica is repaired");
  FR(fr_plan_destroy(rplan));
  hipFree(d_dpay), hipFree(d_dsums), hipFree(d_dbm);
  free(o_dpay), free(g_dpay), free(g_rep);

  FR(fr_plan_destroy(plan));
  HIP(hipStreamDestroy(s));
  hipFree(d_src), hipFree(d_rep), hipFree(d_dst), hipFree(d_pay), hipFree(d_sums);
  hipFree(d_csum), hipFree(d_bm), hipFree(d_diff), hipFree(d_nbad), hipFree(d_ndiff);
  free(src), free(o_pay), free(o_sums), free(o_dst), free(o_bm);
  free(g_pay), free(g_sums), free(g_csum), free(g_dst), free(g_bm);
  printf("c abi ok: %llu chunks, %llu payload bytes, chunk %llu located and repaired (%llu delta bytes)\n",
         (unsigned long long)n, (unsigned long long)pb, (unsigned long long)chunk,
         (unsigned long long)dpb);
  return 0;
}
