// Internal declarations shared by the translation units of libfademem.so.
// Not part of the public interface (include/fademem.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "fademem.h"

namespace fademem {

constexpr int kLogCap = 4096;             // merge-log ring capacity (entries)
constexpr int kMaxPlanFrames = 4;         // frames one fused update plan covers
constexpr int64_t kMaxBudget = 1023;      // schedule runs in one 1024-thread block
constexpr int kMaxLayersPerLaunch = 64;   // layer pointers passed as kernel arguments
constexpr int64_t kMaxPosition = int64_t(1) << 40;
constexpr int64_t kMaxTokens = int64_t(1) << 30;

// bf16 attention work split.  A workgroup (8 waves x 32 queries) runs one
// query tile's key range, or part of it: when the tiles do not fill whole
// rounds of resident workgroups, the remaining tiles are split along the key
// axis between workgroups, each part leaves its partial result (unnormalised
// O, row max and row sums) in a scratch slot, and a second kernel merges the
// two parts of each split tile.  At most kSkMaxGroups workgroups per launch,
// two scratch slots per workgroup.
constexpr int kAttnThreads = 512;        // threads per workgroup (8 waves)
constexpr int kAttnQueries = 256;        // queries per workgroup (32 per wave)
constexpr int kSkMaxGroups = 256;        // workgroups of one launch at most (one per CU)
__host__ __device__ constexpr size_t attend_slot_floats(int head_dim) {
  // O of every query, then the row max and the partial row sum of every
  // (thread, 32-query block).
  return size_t(kAttnQueries) * size_t(head_dim) + 4 * size_t(kAttnQueries);
}
__host__ __device__ constexpr size_t attend_ws_bytes(int head_dim) {
  return 2 * size_t(kSkMaxGroups) * attend_slot_floats(head_dim) * sizeof(float);
}

// fp32 attention work split: a workgroup takes kF32Queries queries of one
// head over a range of key tiles; when the key axis is cut into several
// ranges, each leaves its partial result (unnormalised O, row max and row
// sum per query) in a slot and a second kernel combines them.  At most
// kF32MaxParts slots per call.
constexpr int kF32Queries = 64;
constexpr int kF32MaxParts = 512;
__host__ __device__ constexpr size_t f32_part_floats(int head_dim) {
  return size_t(kF32Queries) * size_t(head_dim + 2);
}
__host__ __device__ constexpr size_t f32_ws_bytes(int head_dim) {
  return size_t(kF32MaxParts) * f32_part_floats(head_dim) * sizeof(float);
}

// Device-resident header at the start of the pool.  Written only by the
// library's kernels; the host reads it back for merge_log.
struct DevHeader {
  int64_t merges_total;   // consolidations run (length of the merge log)
  int64_t anchor_merges;  // of which anchor merges (no K/V work)
};

// Data program of one fused update (F sequential Algorithm S1 updates),
// written by the plan kernel and executed element by element by the data
// kernel.  A value reference is an old entry's slot, a frame of the
// caller's chunk, or the result of an earlier merge of the same update.
enum : int32_t { kRefSlot = 0, kRefFrame = 1, kRefResult = 2 };
struct UpdatePlan {
  int32_t n_ar;                          // merges that compute K, V (in order)
  int32_t n_out;                         // entries to store
  int32_t a_kind[kMaxPlanFrames], a_idx[kMaxPlanFrames];  // older operand of merge k
  int32_t b_kind[kMaxPlanFrames], b_idx[kMaxPlanFrames];  // newer operand of merge k
  double wa[kMaxPlanFrames], wb[kMaxPlanFrames];          // weights of merge k
  int32_t o_kind[2 * kMaxPlanFrames], o_idx[2 * kMaxPlanFrames];
  int32_t o_slot[2 * kMaxPlanFrames];    // destination slot of each stored entry
};

// Pool layout.  The memory's metadata is kept twice (copies 0 and 1): a
// consolidation reads the current copy and writes the other one, so the
// many blocks of the merge kernel that all derive the schedule decision
// from the metadata never race with the block that updates it.  Arrays are
// indexed by logical entry (0 = oldest); order[] maps logical entry -> KV
// slot and is a permutation of the slots whose first `count` elements are
// the live entries' slots (the rest are free), so compaction never moves KV.
struct Layout {
  int64_t slots;          // M + max(1, stage_frames)
  size_t off_first[2];    // int64[slots]
  size_t off_pos_sum[2];  // int64[slots]
  size_t off_span[2];     // int64[slots]
  size_t off_order[2];    // int32[slots]
  size_t off_log;         // int32[kLogCap]
  size_t off_prog;        // UpdatePlan of the last fused update
  size_t meta_bytes;      // multiple of 256
  size_t elt;             // bytes per element
  size_t blk_bytes;       // N*H*D*elt: one K (or V) block
  size_t blk_stride;      // blk_bytes rounded up to 256
  size_t row_elems;       // H*D: elements per token row
  size_t off_ws;          // attention scratch, after the KV region
  size_t ws_bytes;        // attend_ws_bytes(D) for bf16, f32_ws_bytes(D) for fp32
  size_t off_view;        // RoPE views: per layer, one rotated K block per view position (= logical entry)
  size_t view_bytes;      // 0 when rope_pairs = 0
  size_t total;           // off_view + view_bytes
};

int compute_layout(const fademem_config* cfg, Layout* lay);

// Address of layer l, slot s, kind kv (0 = K, 1 = V) inside the KV region.
__host__ __device__ inline size_t kv_offset(const Layout& lay, int64_t layer, int64_t slot, int kv) {
  return lay.meta_bytes + ((size_t(layer) * lay.slots + size_t(slot)) * 2 + kv) * lay.blk_stride;
}

// Attention launchers (attend_bf16.hip, attend_f32.hip).  All pointers are
// device pointers.  The exposed keys are entries e = 0..n_entries-1 of N
// rows each, then the current chunk's cur_tokens rows.  Entry e's K rows
// start at k_base + k_order[e] * k_stride (k_order NULL: the identity) and
// its V rows at v_base + v_order[e] * v_stride; a row is [H][D].  For the
// memory as stored, k_base is the layer's slot 0 K block, v_base its V
// block, both orders the slot table and both strides the slot stride; a
// re-indexed K view or staged frames only change the tables.
struct AttendArgs {
  const void* q;
  void* out;
  float* lse;
  const char* k_base;
  const int32_t* k_order;     // logical -> K block index (NULL: e)
  size_t k_stride;
  const char* v_base;
  const int32_t* v_order;     // logical -> V block index
  size_t v_stride;
  const void* k_cur;
  const void* v_cur;
  int64_t n_entries;          // entries exposed from memory
  int64_t tokens_per_block;   // N
  int64_t cur_tokens;         // rows of the current chunk
  int64_t q_tokens;
  float* ws;                  // attention scratch: 2*kSkMaxGroups slots (bf16), kF32MaxParts slots (fp32)
  int heads;
  int head_dim;
  float scale;
};

hipError_t launch_attend_bf16(const AttendArgs& a, hipStream_t stream);
hipError_t launch_attend_f32(const AttendArgs& a, hipStream_t stream);

}  // namespace fademem
