// Restore planner for data x tensor x pipeline parallel layouts with ZeRO
// sharding (Section III-A: DP, PP, TP, ZeRO/FSDP and their combination;
// Section III-E: restoration for vanilla DP, for ZeRO/FSDP, and for
// combinations of data and model parallelism; Section III-D stage 3: the
// controller picks the device whose state is used).
//
// Layout (the paper fixes none of this; readings):
//   world = TP * DP * PP ranks; rank = tp + TP * (dp + DP * pp)  (tensor
//   parallel fastest, then data parallel, then pipeline).
//   The data-parallel group of a (tp, pp) slice is split into R = DP / S
//   replica groups of S ranks: dp = shard + S * replica.  Stage 0 (vanilla
//   DP) requires S = 1.  Stages 1 and 2 shard the optimizer state (fp32
//   master, Adam m and v) S ways and keep full bf16 parameters; stage 3 also
//   shards the parameters.
//   A slice's tensors are flattened in order into N elements, padded to a
//   multiple of 8 * S, and shard s owns elements [s * E, (s + 1) * E),
//   E = N_pad / S.  Padding elements exist in every array and hold zeros.
//   Ranks with the same (tp, pp, shard) hold identical state: they are each
//   other's replicas.  A failed rank is restored from a live replica; if none
//   is live, only a checkpoint can restore it.
#include <algorithm>
#include <cstdint>
#include <new>
#include <vector>

#include "flashrestore.h"

namespace {

bool layout_ok(const fr_layout3d* L) {
  if (!L || L->tp == 0 || L->pp == 0 || L->dp == 0 || L->shard == 0) return false;
  if (L->dp % L->shard != 0 || L->zero_stage > 3) return false;
  if (L->zero_stage == 0 && L->shard != 1) return false;
  const uint64_t world = uint64_t(L->tp) * L->dp * L->pp;
  return world <= 0x7FFFFFFFull;
}

uint32_t world_of(const fr_layout3d* L) { return L->tp * L->dp * L->pp; }

struct Coords {
  uint32_t tp, pp, dp, shard, replica;
};

Coords coords_of(const fr_layout3d* L, uint32_t rank) {
  Coords c;
  c.tp = rank % L->tp;
  c.dp = (rank / L->tp) % L->dp;
  c.pp = rank / (L->tp * L->dp);
  c.shard = c.dp % L->shard;
  c.replica = c.dp / L->shard;
  return c;
}

// Replica class of a rank: ranks holding identical state.
uint32_t class_of(const fr_layout3d* L, uint32_t rank) {
  const Coords c = coords_of(L, rank);
  return (c.pp * L->tp + c.tp) * L->shard + c.shard;
}

}  // namespace

extern "C" int fr_layout_rank_coords(const fr_layout3d* L, uint32_t rank, uint32_t* coords) {
  if (!layout_ok(L) || !coords) return FR_E_INVAL;
  if (rank >= world_of(L)) return FR_E_RANGE;
  const Coords c = coords_of(L, rank);
  coords[0] = c.tp;
  coords[1] = c.pp;
  coords[2] = c.dp;
  coords[3] = c.shard;
  coords[4] = c.replica;
  return FR_OK;
}

extern "C" int fr_layout_donors(const fr_layout3d* L, const uint8_t* failed, int32_t* donor) {
  if (!layout_ok(L) || !failed || !donor) return FR_E_INVAL;
  const uint32_t world = world_of(L);
  const uint32_t classes = L->tp * L->pp * L->shard;
  std::vector<std::vector<uint32_t>> live;
  std::vector<uint32_t> next;
  try {
    live.resize(classes);
    next.assign(classes, 0);
  } catch (const std::bad_alloc&) {
    return FR_E_NOMEM;
  }
  for (uint32_t r = 0; r < world; r++)
    if (!failed[r]) live[class_of(L, r)].push_back(r);
  // failed ranks of a class are spread over its live ranks in rank order
  for (uint32_t r = 0; r < world; r++) {
    donor[r] = -1;
    if (!failed[r]) continue;
    const uint32_t k = class_of(L, r);
    if (live[k].empty()) continue;
    donor[r] = int32_t(live[k][next[k]++ % live[k].size()]);
  }
  return FR_OK;
}

extern "C" int fr_layout_state_table(const fr_layout3d* L, uint32_t rank, const uint64_t* numel,
                                     uint32_t n_tensors, fr_tensor_desc* table, uint32_t cap,
                                     uint32_t* n_entries, uint64_t* arena_bytes) {
  if (!layout_ok(L) || !n_entries || !arena_bytes || (n_tensors && !numel)) return FR_E_INVAL;
  if (rank >= world_of(L)) return FR_E_RANGE;
  const Coords c = coords_of(L, rank);
  std::vector<fr_tensor_desc> out;
  uint64_t off = 0;
  auto add = [&](uint64_t n, uint32_t dtype, int32_t derive) {
    fr_tensor_desc d{};
    d.src_offset = d.dst_offset = off;
    d.numel = n;
    d.dtype = dtype;
    d.derive_from = derive;
    out.push_back(d);
    const uint64_t nb = n * (dtype == FR_F32 ? 4 : 2);
    off += (nb + 15) & ~uint64_t(15);
    return int32_t(out.size() - 1);
  };
  try {
    if (L->zero_stage == 0) {
      // per tensor: bf16 param (rounded from its master), fp32 master, m, v
      for (uint32_t k = 0; k < n_tensors; k++) {
        if (numel[k] > (uint64_t(1) << 40)) return FR_E_RANGE;
        const int32_t p = int32_t(out.size());
        add(numel[k], FR_BF16, p + 1);
        add(numel[k], FR_F32, -1);
        add(numel[k], FR_F32, -1);
        add(numel[k], FR_F32, -1);
      }
    } else {
      uint64_t n = 0;
      for (uint32_t k = 0; k < n_tensors; k++) {
        if (numel[k] > (uint64_t(1) << 40)) return FR_E_RANGE;
        n += numel[k];
      }
      const uint64_t unit = 8ull * L->shard;
      const uint64_t npad = (n + unit - 1) / unit * unit;
      const uint64_t e = npad / L->shard;
      const uint64_t lo = c.shard * e;
      // entries: [param before shard] [param shard] [param after shard]
      //          [master shard] [m shard] [v shard]; stage 3 keeps only the
      //          parameter shard.  The parameter shard is the master shard
      //          rounded to bf16.
      const int32_t master_index = L->zero_stage == 3 ? 1 : 3;
      if (L->zero_stage == 3) {
        add(e, FR_BF16, master_index);
      } else {
        add(lo, FR_BF16, -1);
        add(e, FR_BF16, master_index);
        add(npad - lo - e, FR_BF16, -1);
      }
      add(e, FR_F32, -1);
      add(e, FR_F32, -1);
      add(e, FR_F32, -1);
    }
  } catch (const std::bad_alloc&) {
    return FR_E_NOMEM;
  }
  *n_entries = uint32_t(out.size());
  *arena_bytes = off;
  if (out.size() > cap) return table ? FR_E_RANGE : FR_OK;  // size query with table = NULL
  if (table) std::copy(out.begin(), out.end(), table);
  return FR_OK;
}
