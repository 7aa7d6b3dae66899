// Target tokens at every tree node for verification at temperature T
// (Tables 3-4 report T = 1). With T > 0 one token is drawn per node from
// softmax(logits / T) by inversion with a caller-supplied uniform u: the
// smallest token index whose cumulative probability, in vocabulary order,
// exceeds u. With T = 0 the token is the argmax (lowest index on ties). Nodes
// whose root paths carry the same draft tokens share one draw, that of the
// lowest-index such node, so that a tree repeating a context stays exact
// under the longest-accepted-path rule that follows.
//
// One workgroup per tree node. It first finds the node's representative from
// the request's parent and token arrays (staged in LDS), then streams the
// representative's logits row once: every wave reduces 2048 (bf16) or 1024
// (fp32) consecutive logits per step to a (max, sum of exp) pair, or to
// (max, first index of the max) for T = 0, kept in LDS per step. The loads of
// two of a wave's steps are issued together, before either is reduced, and
// the first of them go out before the representative search: a node is
// nearly always its own representative, and otherwise they are issued again
// for the representative's row. Wave 0 then scans the step sums in
// vocabulary order, finds the step where the running sum crosses u times the
// total, and re-reads only that step to find the token inside it. Wave
// reductions and scans run on DPP and the lane-pair swaps, not through LDS.
// The row is read from HBM once; the cost is one pass of loads plus one
// exponential per logit.
#include "launchers.h"

namespace d2sd {

namespace {

constexpr int kSampleThreads = 256;
constexpr int kSampleWaves = kSampleThreads / kWave;
constexpr int kLoadsPerStep = 4;                                   // 16-byte loads per lane per step
constexpr int kResident = 2;                                       // steps per wave whose loads are in flight together
constexpr int kMaxSteps = D2SD_MAX_VOCAB / (kWave * kLoadsPerStep * 4);   // fp32 steps hold the fewest logits
constexpr int kMaxNodes = D2SD_MAX_B + D2SD_MAX_B * (D2SD_MAX_B - 1) / 2;   // 2080
constexpr int kNoIndex = 0x7fffffff;

template <int DT>
struct Logits;

// The logits of elements start .. start + kVec - 1, still packed; elements at
// or past V read as -inf. load_elems loads element by element at indices
// clamped into the row, with no branch, so all loads of a step are issued
// before any is used; load_raw takes one 16-byte load when the row is aligned
// and the chunk lies inside it.
template <>
struct Logits<D2SD_BF16> {
  static constexpr int kVec = 8;
  __device__ static __forceinline__ uint4 load_raw(const void* row, long long start, int V, bool vec_ok) {
    const uint16_t* r = static_cast<const uint16_t*>(row);
    if (vec_ok && start + kVec <= V) return *reinterpret_cast<const uint4*>(r + start);
    return load_elems(row, start, V);
  }
  __device__ static __forceinline__ uint4 load_elems(const void* row, long long start, int V) {
    const uint16_t* r = static_cast<const uint16_t*>(row);
    uint32_t e[kVec];
#pragma unroll
    for (int i = 0; i < kVec; ++i) e[i] = r[min(start + i, (long long)V - 1)];
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (start + 2 * i < V ? e[2 * i] : 0xff80u) | ((start + 2 * i + 1 < V ? e[2 * i + 1] : 0xff80u) << 16);
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
  __device__ static __forceinline__ void unpack(const uint4& x, float* v) {
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
};

template <>
struct Logits<D2SD_F32> {
  static constexpr int kVec = 4;
  __device__ static __forceinline__ uint4 load_raw(const void* row, long long start, int V, bool vec_ok) {
    const float* r = static_cast<const float*>(row);
    if (vec_ok && start + kVec <= V) return *reinterpret_cast<const uint4*>(r + start);
    return load_elems(row, start, V);
  }
  __device__ static __forceinline__ uint4 load_elems(const void* row, long long start, int V) {
    const float* r = static_cast<const float*>(row);
    float e[kVec];
#pragma unroll
    for (int i = 0; i < kVec; ++i) e[i] = r[min(start + i, (long long)V - 1)];
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < kVec; ++i) w[i] = __float_as_uint(start + i < V ? e[i] : -INFINITY);
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
  __device__ static __forceinline__ void unpack(const uint4& x, float* v) {
    v[0] = __uint_as_float(x.x); v[1] = __uint_as_float(x.y);
    v[2] = __uint_as_float(x.z); v[3] = __uint_as_float(x.w);
  }
};

template <int DT>
__device__ __forceinline__ void load_logits(const void* row, long long start, int V, bool vec_ok, float* v) {
  Logits<DT>::unpack(Logits<DT>::load_raw(row, start, V, vec_ok), v);
}

// Cross-lane reductions and scans on DPP (inside rows of 16 lanes) and the
// lane-pair swaps (across rows): register to register, with no LDS round trip
// per level. Every lane of a reduction combines the same operands in the same
// order, so all lanes end with identical bits.
constexpr int kQuadSwap1 = 0xB1;      // DPP quad_perm [1,0,3,2]
constexpr int kQuadSwap2 = 0x4E;      // DPP quad_perm [2,3,0,1]
constexpr int kRowMirror = 0x140;     // lane i <- lane 15 - i of its row
constexpr int kRowHalfMirror = 0x141; // lane i <- lane 7 - i of its half row
constexpr int kRowShr = 0x110;        // + n: lane i <- lane i - n of its row
constexpr int kRowBcast15 = 0x142;    // lane 15 of a row -> every lane of the next row
constexpr int kRowBcast31 = 0x143;    // lane 31 -> every lane of rows 2 and 3

// Lanes without a source lane, or outside the row mask, return `old`.
template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ uint32_t dpp(uint32_t old, uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)x, CTRL, ROW_MASK, 0xf, false);
}

template <typename Op>
__device__ __forceinline__ uint32_t wave_reduce(uint32_t x, Op op) {
  x = op(x, dpp<kQuadSwap1>(x, x));
  x = op(x, dpp<kQuadSwap2>(x, x));
  x = op(x, dpp<kRowHalfMirror>(x, x));
  x = op(x, dpp<kRowMirror>(x, x));
  const auto r16 = __builtin_amdgcn_permlane16_swap(x, x, false, false);   // {lane with bit 4 clear, set}
  x = op(r16[0], r16[1]);
  const auto r32 = __builtin_amdgcn_permlane32_swap(x, x, false, false);   // {lane with bit 5 clear, set}
  return op(r32[0], r32[1]);
}

__device__ __forceinline__ float wave_max(float x) {
  return __uint_as_float(wave_reduce(__float_as_uint(x), [](uint32_t a, uint32_t b) {
    return __float_as_uint(fmaxf(__uint_as_float(a), __uint_as_float(b)));
  }));
}

__device__ __forceinline__ float wave_sum(float x) {
  return __uint_as_float(wave_reduce(__float_as_uint(x), [](uint32_t a, uint32_t b) {
    return __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
  }));
}

__device__ __forceinline__ int wave_min(int x) {
  return (int)wave_reduce((uint32_t)x, [](uint32_t a, uint32_t b) { return (uint32_t)min((int)a, (int)b); });
}

// Inclusive prefix sum over the lanes of a wave, in lane order: a
// Hillis-Steele scan inside each row of 16, then the totals of rows 0 and 2
// into rows 1 and 3, then the total of rows 0-1 into rows 2 and 3.
__device__ __forceinline__ float wave_inclusive_scan(float x) {
  x += __uint_as_float(dpp<kRowShr + 1>(0u, __float_as_uint(x)));
  x += __uint_as_float(dpp<kRowShr + 2>(0u, __float_as_uint(x)));
  x += __uint_as_float(dpp<kRowShr + 4>(0u, __float_as_uint(x)));
  x += __uint_as_float(dpp<kRowShr + 8>(0u, __float_as_uint(x)));
  x += __uint_as_float(dpp<kRowBcast15, 0xa>(0u, __float_as_uint(x)));
  x += __uint_as_float(dpp<kRowBcast31, 0xc>(0u, __float_as_uint(x)));
  return x;
}

// Value of x in lane `src` (uniform over the wave).
__device__ __forceinline__ float lane_value(float x, int src) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), src));
}
__device__ __forceinline__ int lane_value(int x, int src) { return __builtin_amdgcn_readlane(x, src); }

__device__ __forceinline__ int first_lane(uint64_t mask) { return mask ? __ffsll((long long)mask) - 1 : -1; }

// The exponent offset of a step whose max is m: the product rounded on its
// own, never fused, so that the per-step sums and the later rescaling see the
// same value.
__device__ __forceinline__ float step_offset(float m, float k2) { return __fmul_rn(m, k2); }

// 2^(offset(ms) - offset(mx)): rescales weights taken against a step's max to
// the row's max. Weights exp2(l k2 - offset(ms)) times this factor equal
// exp2(l k2 - offset(mx)) for every step, so all steps share one reference.
__device__ __forceinline__ float step_scale(float ms, float mx, float k2) {
  return __builtin_amdgcn_exp2f(step_offset(ms, k2) - step_offset(mx, k2));
}

// Token index of lane element i of a step: load k = i / VEC covers
// kWave * VEC consecutive logits, lane-major.
template <int VEC>
__device__ __forceinline__ int step_index(int s, int lane, int i) {
  return s * (kWave * kLoadsPerStep * VEC) + (i / VEC) * (kWave * VEC) + lane * VEC + (i % VEC);
}

// Issue the loads of kResident whole steps of a wave (steps s0, s0 + waves,
// ...) of an aligned row: plain 16-byte loads under a wave-uniform bound.
template <int DT>
__device__ __forceinline__ void load_full(uint4 (&raw)[kResident][kLoadsPerStep], const void* rowp, int s0,
                                          int n_full, int lane) {
  constexpr int VEC = Logits<DT>::kVec;
  const uint4* r = static_cast<const uint4*>(rowp);
#pragma unroll
  for (int j = 0; j < kResident; ++j) {
    const int s = s0 + j * kSampleWaves;
    if (s < n_full) {
#pragma unroll
      for (int k = 0; k < kLoadsPerStep; ++k) raw[j][k] = r[step_index<VEC>(s, lane, k * VEC) / VEC];
    }
  }
}

// One step's (max, sum of exp relative to it) or, for T = 0, (max, first
// index of the max), kept in LDS by lane 0.
template <int DT>
__device__ __forceinline__ void reduce_step(const uint4 (&raw)[kLoadsPerStep], int s, int lane, int greedy,
                                            float k2, float* s_m, float* s_x) {
  constexpr int VEC = Logits<DT>::kVec;
  constexpr int NE = kLoadsPerStep * VEC;
  float v[NE];
#pragma unroll
  for (int k = 0; k < kLoadsPerStep; ++k) Logits<DT>::unpack(raw[k], v + k * VEC);
  float lm = v[0];
#pragma unroll
  for (int i = 1; i < NE; ++i) lm = fmaxf(lm, v[i]);
  const float m = wave_max(lm);
  float x;
  if (greedy) {
    int first = kNoIndex;                    // elements of a lane ascend with i
#pragma unroll
    for (int i = NE - 1; i >= 0; --i)
      if (v[i] == m) first = step_index<VEC>(s, lane, i);
    x = __int_as_float(m == -INFINITY ? kNoIndex : wave_min(first));
  } else {
    float sum = 0.0f;
    if (m != -INFINITY) {
      const float moff = step_offset(m, k2);
#pragma unroll
      for (int i = 0; i < NE; ++i) sum += __builtin_amdgcn_exp2f(fmaf(v[i], k2, -moff));
    }
    x = wave_sum(sum);
  }
  if (lane == 0) {
    s_m[s] = m;
    s_x[s] = x;
  }
}

template <int DT>
__global__ __launch_bounds__(kSampleThreads) void sample_targets_kernel(
    const int* __restrict__ node_indptr, int total_nodes, int max_nodes, const int* __restrict__ parent,
    const int* __restrict__ draft, int V, const void* __restrict__ logits, int greedy, float k2,
    const float* __restrict__ uniform, int* __restrict__ rep_out, int* __restrict__ tokens_out) {
  constexpr int VEC = Logits<DT>::kVec;
  constexpr int NE = kLoadsPerStep * VEC;       // logits per lane per step
  constexpr int SE = kWave * NE;                // logits per step
  constexpr size_t kEltBytes = DT == D2SD_BF16 ? 2 : 4;
  __shared__ float s_m[kMaxSteps];              // per-step max
  __shared__ float s_x[kMaxSteps];              // per-step sum of exp (T > 0) or first argmax index (T = 0)
  __shared__ short s_par[kMaxNodes];
  __shared__ int s_tok[kMaxNodes];
  __shared__ int s_path[D2SD_MAX_B];            // tokens of this node's root path, leaf first
  __shared__ int s_walk[2];                     // path length (-1: no root within bounds), root
  __shared__ int s_best[kSampleWaves];

  const int b = blockIdx.x / max_nodes;
  const int c = blockIdx.x % max_nodes;
  const int t = threadIdx.x, lane = t % kWave, w = t / kWave;
  const int base = clampi(node_indptr[b], 0, total_nodes);
  const int Nb = clampi(node_indptr[b + 1] - base, 0, min(kMaxNodes, total_nodes - base));
  if (c >= Nb) return;

  // ---- representative: the lowest-index node with the same root path tokens
  for (int x = t; x <= c; x += kSampleThreads) {
    int par = parent[base + x];
    if (par < 0 || par >= x) par = -1;          // parents precede children
    s_par[x] = (short)par;
    s_tok[x] = draft[base + x];
  }
  // The node is usually its own representative: the first loads of its row go
  // out now (after the staging above, whose wait would otherwise include
  // them) and are in flight during the search below.
  const int n_steps = ceil_div(V, SE);
  const int n_whole = V / SE;                   // steps lying wholly inside the row
  const void* row_c = static_cast<const char*>(logits) + (size_t)(base + c) * (size_t)V * kEltBytes;
  const bool vec_ok_c = ((size_t)(base + c) * (size_t)V) % VEC == 0;   // the row starts 16-byte aligned
  uint4 raw[kResident][kLoadsPerStep];
  load_full<DT>(raw, row_c, w, vec_ok_c ? n_whole : 0, lane);
  __syncthreads();
  if (t == 0) {
    int x = c, d = 0;
    while (s_par[x] >= 0 && d < D2SD_MAX_B) {
      s_path[d++] = s_tok[x];
      x = s_par[x];
    }
    s_walk[0] = s_par[x] >= 0 ? -1 : d;
    s_walk[1] = x;
  }
  __syncthreads();
  const int depth = s_walk[0], root = s_walk[1];
  int best = c;
  if (depth >= 0) {
    for (int m = t; m < c; m += kSampleThreads) {
      int x = m;
      bool ok = true;
      for (int i = 0; i < depth && ok; ++i) {
        const int px = s_par[x];
        ok = px >= 0 && s_tok[x] == s_path[i];
        x = px;
      }
      if (ok && x == root) best = min(best, m);   // x == root implies x is a root
    }
  }
  best = wave_min(best);
  if (lane == 0) s_best[w] = best;
  __syncthreads();
  int rep = s_best[0];
#pragma unroll
  for (int i = 1; i < kSampleWaves; ++i) rep = min(rep, s_best[i]);

  // ---- one pass over the representative's row: per-step (max, sum) or (max, index)
  const size_t row = (size_t)(base + rep);
  const void* rowp = static_cast<const char*>(logits) + row * (size_t)V * kEltBytes;
  const bool vec_ok = (row * (size_t)V) % VEC == 0;
  // A wave takes steps w, w + 4, ...: the whole steps of an aligned row in
  // batches of kResident whose loads are issued together, then the rest (a
  // ragged last step, or every step of an unaligned row) element by element.
  const int n_full = vec_ok ? n_whole : 0;
  if (rep != c) load_full<DT>(raw, rowp, w, n_full, lane);
  for (int s0 = w; s0 < n_full; s0 += kSampleWaves * kResident) {
    if (s0 != w) load_full<DT>(raw, rowp, s0, n_full, lane);
#pragma unroll
    for (int j = 0; j < kResident; ++j) {
      const int s = s0 + j * kSampleWaves;
      if (s < n_full) reduce_step<DT>(raw[j], s, lane, greedy, k2, s_m, s_x);
    }
  }
  for (int s = w; s < n_steps; s += kSampleWaves) {
    if (s < n_full) continue;
    uint4 tail[kLoadsPerStep];
#pragma unroll
    for (int k = 0; k < kLoadsPerStep; ++k)
      tail[k] = Logits<DT>::load_elems(rowp, (long long)step_index<VEC>(s, lane, k * VEC), V);
    reduce_step<DT>(tail, s, lane, greedy, k2, s_m, s_x);
  }
  __syncthreads();
  if (w != 0) return;

  // ---- wave 0: the row's max, then the token
  float mx = -INFINITY;
  for (int s = lane; s < n_steps; s += kWave) mx = fmaxf(mx, s_m[s]);
  mx = wave_max(mx);
  int token = -1;
  if (mx == -INFINITY) {
    // no finite logit: -1
  } else if (greedy) {
    int first = kNoIndex;                      // lowest step reaching the max, then its first index
    for (int s = lane; s < n_steps; s += kWave)
      if (s_m[s] == mx) first = min(first, s);
    first = wave_min(first);
    token = __float_as_int(s_x[first]);
  } else {
    // step weights a_s = sum_s * 2^((m_s - mx) k2); running sums in step order
    auto weight = [&](int s) {
      return s < n_steps && s_x[s] > 0.0f ? s_x[s] * step_scale(s_m[s], mx, k2) : 0.0f;
    };
    float total = 0.0f;
    for (int s0 = 0; s0 < n_steps; s0 += kWave) total += lane_value(wave_inclusive_scan(weight(s0 + lane)), kWave - 1);
    const float target = uniform[row] * total;
    int sel = -1;
    float before = 0.0f;                       // running sum before step sel
    float carry = 0.0f;
    for (int s0 = 0; s0 < n_steps && sel < 0; s0 += kWave) {
      const float a = weight(s0 + lane);
      const float cum = carry + wave_inclusive_scan(a);
      const int f = first_lane(__ballot(cum > target));
      if (f >= 0) {
        sel = s0 + f;
        before = lane_value(cum - a, f);
      }
      carry = lane_value(cum, kWave - 1);
    }
    int last_pos = -1;                         // rounding left no crossing: last step of positive weight
    if (sel < 0) {
      for (int s = lane; s < n_steps; s += kWave)
        if (weight(s) > 0.0f) last_pos = max(last_pos, s);
      sel = -wave_min(-last_pos);
      before = 0.0f;
    }
    // inside step sel: weights relative to its own max, as in the pass above.
    // sel < 0 only when every step's sum is NaN (a NaN logit): token -1.
    if (sel >= 0) {
      float v[NE];
#pragma unroll
      for (int k = 0; k < kLoadsPerStep; ++k)
        load_logits<DT>(rowp, (long long)step_index<VEC>(sel, lane, k * VEC), V, vec_ok, v + k * VEC);
      const float ms = s_m[sel];
      const float moff = step_offset(ms, k2);
      const float scale = step_scale(ms, mx, k2);
      const float rel = last_pos >= 0 ? INFINITY : (target - before) / scale;   // threshold in step units
      float run = 0.0f;
      int last = -1;
#pragma unroll
      for (int k = 0; k < kLoadsPerStep; ++k) {
        float incl[VEC];
        float acc = 0.0f;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const float we = __builtin_amdgcn_exp2f(fmaf(v[k * VEC + e], k2, -moff));
          acc += we;
          incl[e] = acc;
          if (we > 0.0f) last = step_index<VEC>(sel, lane, k * VEC + e);
        }
        const float lane_incl = wave_inclusive_scan(acc);
        const float lane_excl = run + lane_incl - acc;
        int hit = -1;
#pragma unroll
        for (int e = VEC - 1; e >= 0; --e)
          if (lane_excl + incl[e] > rel) hit = e;
        const int f = first_lane(__ballot(hit >= 0));
        if (f >= 0 && token < 0) token = step_index<VEC>(sel, f, k * VEC + lane_value(hit, f));
        run += lane_value(lane_incl, kWave - 1);
      }
      if (token < 0) token = -wave_min(-last);  // last token of positive weight in the step
    }
  }
  if (lane == 0) {
    tokens_out[base + c] = token;
    if (rep_out) rep_out[base + c] = rep;
  }
}

}  // namespace

hipError_t launch_sample_targets(int batch, const int* node_indptr, int total_nodes, int max_nodes,
                                 const int* parent, const int* draft, int vocab, int dtype, const void* logits,
                                 float temperature, const float* uniform, int* context_rep, int* tokens,
                                 hipStream_t stream) {
  const int greedy = temperature == 0.0f;
  const float k2 = greedy ? 0.0f : (float)(1.4426950408889634 / (double)temperature);   // log2(e) / T
  const dim3 grid((unsigned)((long long)batch * max_nodes));
  if (dtype == D2SD_BF16)
    hipLaunchKernelGGL(sample_targets_kernel<D2SD_BF16>, grid, dim3(kSampleThreads), 0, stream, node_indptr,
                       total_nodes, max_nodes, parent, draft, vocab, logits, greedy, k2, uniform, context_rep,
                       tokens);
  else
    hipLaunchKernelGGL(sample_targets_kernel<D2SD_F32>, grid, dim3(kSampleThreads), 0, stream, node_indptr,
                       total_nodes, max_nodes, parent, draft, vocab, logits, greedy, k2, uniform, context_rep,
                       tokens);
  return hipGetLastError();
}

}  // namespace d2sd
