// Internal definitions shared by the libd2sd translation units (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "d2sd.h"

namespace d2sd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }
__host__ __device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Bits [lo, hi) of a bit set restricted to word w (bits 32w .. 32w+31).
__device__ __forceinline__ uint32_t range_bits(int lo, int hi, int w) {
  const int a = max(lo, 32 * w) - 32 * w;
  const int e = min(hi, 32 * w + 32) - 32 * w;
  if (a >= e) return 0u;
  const uint32_t ones = (e - a) == 32 ? 0xffffffffu : ((1u << (e - a)) - 1u);
  return ones << a;
}

// Resolved plan of one verify-attention call (host side).
struct AttnPlan {
  int G;             // query heads per KV head
  int waves;         // waves (query tiles) per workgroup: 4, or 12 for the wide bf16 shapes
  bool packed;       // 12 waves over the global tile sequence (several streams per workgroup)
  long long tiles;   // packed: query tiles of all streams (the grid holds ceil(tiles / 12) workgroups)
  int split;         // context tokens per split (multiple of 64)
  int n_ch_max;      // splits of the longest context (>= 1)
  int n_rg_max;      // row groups of the largest request (>= 1)
  long long items;   // batch * hkv * n_ch_max * n_rg_max
  size_t ws_bytes;   // partial-state workspace (0 when n_ch_max == 1)
  float scale;       // softmax scale
};

// ev (nullable events): ev[0] is recorded before the main kernel, ev[1]
// after it, and ev[2] after the split merge; ev[2] is left unrecorded when
// the call launches no merge (the caller then times the main kernel only).
hipError_t launch_cascade_attention(const d2sd_attn_args& a, const AttnPlan& plan, void* ws,
                                    hipStream_t stream, hipEvent_t (&ev)[3]);

hipError_t launch_noncascade_attention(const d2sd_attn_args& a, float scale, hipStream_t stream,
                                       hipEvent_t (&ev)[3]);

// Size of the static device scratch that backs the allocation-free attention
// entry point (split partial states), and its device address on the current
// device (looked up once per device).
constexpr size_t kScratchBytes = 64ull << 20;
hipError_t scratch_address(void** out);

hipError_t launch_merge_state(int rows, int head_dim, const float* o_a, const float* lse_a,
                              const float* o_b, const float* lse_b, float* o_out, float* lse_out,
                              hipStream_t stream);

// Waves (one 32-query column tile each) per workgroup of the bf16 kernel,
// in its two shapes. Four-wave workgroups let three workgroups share a CU,
// so each SIMD runs three independent waves that hide each other's barrier
// and copy waits; twelve-wave workgroups (one per CU, three waves per SIMD)
// share one K/V ring among 384 query rows.
constexpr int kBf16Waves = 4;
constexpr int kBf16WideWaves = 12;

// The packed twelve-wave kernel: at least kPackedMinTiles query tiles per
// stream (so that 12 consecutive tiles span at most three streams), at most
// kPackedMaxBatch requests and kPackedMaxSplit context tokens per split.
constexpr int kPackedMinTiles = 6;
constexpr int kPackedMaxBatch = 2048;
constexpr int kPackedMaxSplit = 16384;

// Rows (queries) per MFMA column tile. A work item's row group is one tile
// per wave: 32 * plan.waves rows (fp32: always 4 waves).
constexpr int kRowsPerTile = 32;

// Split merge: 16 lanes per output row (8 dims each) and kMergeGroups(n)
// groups of them per row, each folding every kMergeGroups-th split; a
// workgroup of 256 threads then takes merge_rows(n) rows, and the grid is
// batch x merge_chunks_per_request(...) workgroups.
__host__ __device__ constexpr int merge_groups(int n_ch_max) { return n_ch_max >= 4 ? 4 : 1; }
__host__ __device__ constexpr int merge_rows(int groups) { return 256 / (16 * groups); }
__host__ __device__ inline long long merge_chunks_per_request(int max_nodes, int hq, int groups) {
  return ((long long)max_nodes * hq + merge_rows(groups) - 1) / merge_rows(groups);
}

}  // namespace d2sd
