// Internal declarations shared by the host sources and the gfx950 kernels.
#pragma once

#include <stdint.h>

#include <vector>

#include "flashrestore.h"

namespace fr {

constexpr uint64_t kNoPayload = ~uint64_t(0);
constexpr uint32_t kNoMaster = 0xFFFFFFFFu;

// One record per global chunk id, uploaded once per plan.  Every kernel reads
// the record of the unit it works on with uniform (scalar) loads.
struct alignas(16) ChunkRec {
  uint64_t src_off;  // chunk start in the sender / replica arena
  uint64_t pay_off;  // chunk start in the payload; kNoPayload for derived entries
  uint64_t dst_off;  // chunk start in the receiver arena
  uint32_t len;      // bytes in this chunk (<= C, even)
  uint32_t master;   // derived chunk j: global id of master chunk 2j; else kNoMaster
};
static_assert(sizeof(ChunkRec) == 32, "ChunkRec is 32 bytes");

// Host-side layout of a validated table.
struct Layout {
  uint64_t C = 0;
  uint64_t n_chunks = 0;
  uint64_t payload_bytes = 0;
  uint64_t state_bytes = 0;
  std::vector<uint64_t> pay_off;     // per entry; kNoPayload for derived
  std::vector<uint64_t> chunk_base;  // n_entries + 1
};

int validate_and_layout(const fr_tensor_desc* table, uint32_t n, uint64_t C, uint64_t src_bytes,
                        uint64_t dst_bytes, Layout* out);

// Launch configuration shared by all kernels.
struct LaunchCfg {
  uint32_t max_grid;  // upper bound on workgroups per launch (grid-stride beyond)
};

// Kernel launchers (kernels.hip).  They assume validated arguments, enqueue
// on `stream` and return the hipError_t of the launches as an int.
int launch_pack(const ChunkRec* chunks, uint32_t n_chunks, const void* src, void* payload,
                fr_chunk_sum* sums, const LaunchCfg& cfg, void* stream);
int launch_checksum(const ChunkRec* chunks, uint32_t n_chunks, const void* base,
                    fr_chunk_sum* sums, const LaunchCfg& cfg, void* stream);
int launch_unpack(const ChunkRec* chunks, const uint32_t* units, uint32_t n_units, uint64_t C,
                  uint64_t bitmap_words, const void* payload, const fr_chunk_sum* sums,
                  void* dst, uint32_t* bitmap, uint64_t* n_bad, const LaunchCfg& cfg,
                  void* stream);
int launch_verify(const ChunkRec* chunks, uint32_t n_chunks, uint64_t bitmap_words,
                  const void* a, const void* b, uint32_t* bitmap, uint64_t* n_diff,
                  fr_chunk_sum* sums_a, fr_chunk_sum* sums_b, const LaunchCfg& cfg,
                  void* stream);

}  // namespace fr

struct fr_plan {
  int device = -1;
  std::vector<fr_tensor_desc> table;
  fr::Layout layout;
  uint64_t src_arena_bytes = 0, dst_arena_bytes = 0;
  fr::ChunkRec* d_chunks = nullptr;  // n_chunks records
  uint32_t* d_units = nullptr;       // unpack work list
  uint32_t n_units = 0;
  fr::LaunchCfg cfg{};
};
