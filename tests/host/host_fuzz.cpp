// Randomised checks of the library's host code, built with AddressSanitizer
// and UndefinedBehaviorSanitizer by tests/test_host_sanitized.py (g++, CPU
// only; no device code is built or run):
//   1. the step-tag tracker and the layout planner under random call
//      sequences, arguments out of range included;
//   2. table validation and layout (fr_layout_query) on random tables,
//      adversarial sizes and offsets included;
//   3. the delta payload layout (fr_delta_layout) against the C oracle's on
//      random tables and lists, and a full list against the full payload.
// The plan of check 3 has its host fields filled directly (no device).
#include <cstdio>
#include <random>
#include <vector>

#include "flashrestore.h"
#include "fr_internal.h"
extern "C" {
#include "fr_oracle.h"
}

// The kernel launchers and tile helpers live in the device source, which is
// not built here; the checks never reach them.
namespace fr {
uint32_t tile_bytes(int) { return 4096; }
uint64_t accumulators_per_chunk(uint64_t, int) { return 1; }
int static_scratch_address(int, void**) { return 1; }
int launch_delta_build(const DeltaBuild&, bool, void*) { return 1; }
int launch_ids_to_bits(const uint32_t*, uint64_t, uint32_t*, uint64_t, void*) { return 1; }
int launch_pack(const SrcUnit*, const SlotTable&, uint32_t, uint64_t, const void*, void*,
                fr_chunk_sum*, const Scratch&, const LaunchCfg&, void*) { return 1; }
int launch_pack_blocks(const SrcUnit*, const PackBlocks&, uint32_t, uint64_t, const void*, void*,
                       fr_chunk_sum*, const Scratch&, const LaunchCfg&, void*) { return 1; }
int launch_block_first(const uint64_t*, uint64_t, uint64_t, uint64_t, uint32_t, uint32_t*, void*) {
  return 1;
}
int launch_unpack_blocks(const UnpackArgs&, const UnpackBlocks&, const LaunchCfg&, void*) { return 1; }
int launch_checksum(const SrcUnit*, const SlotTable&, uint32_t, uint64_t, const void*,
                    fr_chunk_sum*, const Scratch&, const LaunchCfg&, void*) { return 1; }
int launch_unpack(const UnpackArgs&, const LaunchCfg&, void*) { return 1; }
int launch_compare_sums(const fr_chunk_sum*, const fr_chunk_sum*, uint32_t, uint32_t*, uint64_t*,
                        void*) { return 1; }
int launch_unpack_delta(const UnpackDeltaArgs&, const LaunchCfg&, void*) { return 1; }
int launch_verify(const SrcUnit*, const SlotTable&, uint32_t, uint64_t, const void*, const void*,
                  uint32_t*, uint64_t*, fr_chunk_sum*, fr_chunk_sum*, const Scratch&,
                  const LaunchCfg&, void*) { return 1; }
int launch_expand_slots(const uint64_t*, const uint64_t*, uint64_t, uint64_t, uint64_t, uint64_t*,
                        void*) { return 1; }
}  // namespace fr

namespace {

std::mt19937_64 rng(20260);
uint64_t U(uint64_t n) { return n ? rng() % n : 0; }

void tracker_and_planner() {
  for (int it = 0; it < 2000; it++) {
    const uint32_t n = 1 + U(64);
    std::vector<uint32_t> g(n);
    for (auto& x : g) x = U(n + (it % 50 == 0));  // sometimes an invalid group id
    fr_tracker* t = nullptr;
    double now = 0;
    if (fr_tracker_create(n, (it % 3) ? g.data() : nullptr, 0.1 + U(100) / 10.0, now, &t) != FR_OK)
      continue;
    std::vector<uint32_t> ranks(n + 3);
    std::vector<int32_t> donors(n);
    for (int e = 0; e < 200; e++) {
      now += U(1000) / 2000.0;
      const uint32_t r = U(n + 2);
      switch (U(5)) {
        case 0:
        case 1: fr_tracker_heartbeat(t, r, int64_t(U(6)) - 2, now); break;
        case 2: fr_tracker_report_failure(t, r, now); break;
        case 3: {
          fr_decision d;
          fr_tracker_decide(t, now, &d);
          break;
        }
        default: {
          uint32_t k = 0;
          fr_tracker_failed_ranks(t, now, ranks.data(), uint32_t(U(n + 3)), &k);
          fr_tracker_donors(t, now, donors.data());
        }
      }
    }
    fr_tracker_destroy(t);
  }
  for (int it = 0; it < 2000; it++) {
    fr_layout3d L{uint32_t(1 + U(8)), uint32_t(1 + U(4)), uint32_t(1 + U(12)), uint32_t(1 + U(4)),
                  uint32_t(U(5)), 0};
    if (it % 7 == 0) L.tp = 0;
    uint64_t world = uint64_t(L.tp) * L.pp * L.dp;
    if (world == 0) world = 1;
    uint32_t coords[5];
    for (uint32_t r = 0; r < world + 2; r++) fr_layout_rank_coords(&L, r, coords);
    std::vector<uint8_t> failed(world);
    for (auto& f : failed) f = U(3) == 0;
    std::vector<int32_t> donor(world);
    fr_layout_donors(&L, failed.data(), donor.data());
    std::vector<uint64_t> numel(U(6));
    for (auto& x : numel) x = U(100000);
    for (uint32_t r = 0; r < world && r < 16; r++) {
      uint32_t ne = 0;
      uint64_t ab = 0;
      if (fr_layout_state_table(&L, r, numel.data(), uint32_t(numel.size()), nullptr, 0, &ne, &ab) != FR_OK)
        continue;
      std::vector<fr_tensor_desc> tab(ne + 1);
      fr_layout_state_table(&L, r, numel.data(), uint32_t(numel.size()), tab.data(), uint32_t(U(ne + 2)), &ne, &ab);
      fr_layout_state_table(&L, r, numel.data(), uint32_t(numel.size()), tab.data(), ne, &ne, &ab);
      fr_plan_info info;
      std::vector<uint64_t> po(ne + 1), cb(ne + 2);
      fr_layout_query(tab.data(), ne, 1ull << (4 + U(12)), ab, ab, 16ull << U(9), &info, po.data(),
                      cb.data());
    }
  }
}

void table_validation() {
  for (int it = 0; it < 100000; it++) {
    const uint32_t n = U(12);
    std::vector<fr_tensor_desc> t(n);
    const uint64_t arena = 1ull << U(40);
    for (uint32_t k = 0; k < n; k++) {
      fr_tensor_desc& d = t[k];
      const int mode = int(U(10));
      d.numel = mode == 0 ? (1ull << U(64)) : U(1ull << U(20));
      d.dtype = U(10) == 0 ? uint32_t(U(5)) : uint32_t(1 + U(2));
      d.src_offset = mode == 1 ? ~0ull - U(100) : (U(arena) & ~15ull) + (U(20) == 0 ? 8 : 0);
      d.dst_offset = mode == 2 ? ~0ull - U(100) : (U(arena) & ~15ull);
      d.derive_from = U(3) == 0 ? int32_t(U(n + 2)) - 1 : -1;
    }
    for (uint32_t k = 0; k < n; k++)  // sometimes make a derivation consistent
      if (t[k].derive_from >= 0 && uint32_t(t[k].derive_from) < n && U(2)) {
        const uint32_t m = uint32_t(t[k].derive_from);
        t[m].dtype = FR_F32;
        t[m].numel = t[k].numel;
        t[m].derive_from = -1;
      }
    fr_plan_info info;
    std::vector<uint64_t> po(n + 1), cb(n + 2);
    const uint64_t C = U(8) == 0 ? U(1 << 20) : (1ull << (4 + U(27)));
    const uint64_t seg = U(8) == 0 ? U(1 << 22) : (16ull << U(17));  // sometimes invalid
    fr_layout_query(n ? t.data() : nullptr, n, C, arena, arena, seg, &info, po.data(), cb.data());
  }
}

int delta_layout_vs_oracle() {
  int bad = 0;
  for (int it = 0; it < 10000; it++) {
    const uint32_t n = 1 + U(10);
    std::vector<fr_tensor_desc> t(n);
    for (uint32_t k = 0; k < n; k++) {
      t[k].numel = U(4) == 0 ? 0 : 1 + U(1ull << U(16));
      t[k].dtype = uint32_t(1 + U(2));
      t[k].derive_from = -1;
    }
    for (uint32_t k = 0; k + 1 < n; k++)
      if (U(3) == 0 && t[k].derive_from == -1 && t[k + 1].derive_from == -1) {
        t[k].dtype = FR_BF16;
        t[k].derive_from = int32_t(k + 1);
        t[k + 1].dtype = FR_F32;
        t[k + 1].numel = t[k].numel;
      }
    uint64_t off = 0;
    for (uint32_t k = 0; k < n; k++) {
      t[k].src_offset = t[k].dst_offset = off;
      off += (t[k].numel * (t[k].dtype == FR_F32 ? 4 : 2) + 15) & ~15ull;
    }
    const uint64_t C = 1ull << (4 + U(14));
    const uint64_t seg = 16ull << U(10);
    fr_plan p;
    if (fr::validate_and_layout(t.data(), n, C, seg, off, off, &p.layout) != FR_OK) continue;
    p.table = t;
    p.src_arena_bytes = p.dst_arena_bytes = off;
    std::vector<uint32_t> ids;
    for (uint64_t c = 0; c < p.layout.n_chunks; c++)
      if (U(3)) ids.push_back(uint32_t(c));
    uint64_t got = 0, exp = 0;
    if (fr_delta_layout(&p, ids.data(), ids.size(), &got) != FR_OK) return 1;
    std::vector<oro_entry> ot(n);
    for (uint32_t k = 0; k < n; k++)
      ot[k] = oro_entry{t[k].src_offset, t[k].dst_offset, t[k].numel, t[k].dtype, t[k].derive_from};
    std::vector<uint64_t> oo(ids.size() + 1);
    if (oro_delta_layout(ot.data(), n, C, seg, ids.data(), ids.size(), oo.data(), &exp) != 0) return 1;
    if (got != exp) bad++;
    std::vector<uint32_t> all(p.layout.n_chunks);
    for (uint64_t c = 0; c < all.size(); c++) all[c] = uint32_t(c);
    if (fr_delta_layout(&p, all.data(), all.size(), &got) != FR_OK || got != p.layout.payload_bytes) bad++;
  }
  return bad;
}

}  // namespace

int main() {
  tracker_and_planner();
  table_validation();
  const int bad = delta_layout_vs_oracle();
  std::printf("host fuzz: %d delta layout mismatches\n", bad);
  return bad ? 1 : 0;
}
