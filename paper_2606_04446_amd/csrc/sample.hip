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
// (max, first index of the max) for T = 0, kept in LDS per step. Wave 0 then
// scans the step sums in vocabulary order, finds the step where the running
// sum crosses u times the total, and re-reads only that step to find the
// token inside it. The row is read from HBM once; the cost is one pass of
// loads plus one exponential per logit.
#include "launchers.h"

namespace d2sd {

namespace {

constexpr int kSampleThreads = 256;
constexpr int kSampleWaves = kSampleThreads / kWave;
constexpr int kLoadsPerStep = 4;                                   // 16-byte loads per lane per step
constexpr int kMaxSteps = D2SD_MAX_VOCAB / (kWave * kLoadsPerStep * 4);   // fp32 steps hold the fewest logits
constexpr int kMaxNodes = D2SD_MAX_B + D2SD_MAX_B * (D2SD_MAX_B - 1) / 2;   // 2080
constexpr int kNoIndex = 0x7fffffff;

template <int DT>
struct Logits;

template <>
struct Logits<D2SD_BF16> {
  static constexpr int kVec = 8;
  // Eight logits from element `start` on; elements at or past V read as -inf.
  __device__ static __forceinline__ void load(const void* row, long long start, int V, bool vec_ok, float* v) {
    const uint16_t* r = static_cast<const uint16_t*>(row);
    if (vec_ok && start + kVec <= V) {
      const uint4 x = *reinterpret_cast<const uint4*>(r + start);
      const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[2 * i] = __uint_as_float(w[i] << 16);
        v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
      }
    } else {
#pragma unroll
      for (int e = 0; e < kVec; ++e)
        v[e] = start + e < V ? __uint_as_float((uint32_t)r[start + e] << 16) : -INFINITY;
    }
  }
};

template <>
struct Logits<D2SD_F32> {
  static constexpr int kVec = 4;
  __device__ static __forceinline__ void load(const void* row, long long start, int V, bool vec_ok, float* v) {
    const float* r = static_cast<const float*>(row);
    if (vec_ok && start + kVec <= V) {
      const float4 x = *reinterpret_cast<const float4*>(r + start);
      v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
    } else {
#pragma unroll
      for (int e = 0; e < kVec; ++e) v[e] = start + e < V ? r[start + e] : -INFINITY;
    }
  }
};

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off /= 2) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off /= 2) x += __shfl_xor(x, off);
  return x;
}

__device__ __forceinline__ int wave_min(int x) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off /= 2) x = min(x, __shfl_xor(x, off));
  return x;
}

// Inclusive prefix sum over the lanes of a wave, in lane order.
__device__ __forceinline__ float wave_inclusive_scan(float x, int lane) {
#pragma unroll
  for (int off = 1; off < kWave; off *= 2) {
    const float y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  return x;
}

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
  const bool vec_ok = (row * (size_t)V) % VEC == 0;   // the row starts 16-byte aligned
  const int n_steps = ceil_div(V, SE);
  for (int s = w; s < n_steps; s += kSampleWaves) {
    float v[NE];
#pragma unroll
    for (int k = 0; k < kLoadsPerStep; ++k)
      Logits<DT>::load(rowp, (long long)step_index<VEC>(s, lane, k * VEC), V, vec_ok, v + k * VEC);
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
    for (int s0 = 0; s0 < n_steps; s0 += kWave) total += __shfl(wave_inclusive_scan(weight(s0 + lane), lane), kWave - 1);
    const float target = uniform[row] * total;
    int sel = -1;
    float before = 0.0f;                       // running sum before step sel
    float carry = 0.0f;
    for (int s0 = 0; s0 < n_steps && sel < 0; s0 += kWave) {
      const float a = weight(s0 + lane);
      const float cum = carry + wave_inclusive_scan(a, lane);
      const int f = first_lane(__ballot(cum > target));
      if (f >= 0) {
        sel = s0 + f;
        before = __shfl(cum - a, f);
      }
      carry = __shfl(cum, kWave - 1);
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
        Logits<DT>::load(rowp, (long long)step_index<VEC>(sel, lane, k * VEC), V, vec_ok, v + k * VEC);
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
        const float lane_incl = wave_inclusive_scan(acc, lane);
        const float lane_excl = run + lane_incl - acc;
        int hit = -1;
#pragma unroll
        for (int e = VEC - 1; e >= 0; --e)
          if (lane_excl + incl[e] > rel) hit = e;
        const int f = first_lane(__ballot(hit >= 0));
        if (f >= 0 && token < 0) token = step_index<VEC>(sel, f, k * VEC + __shfl(hit, f));
        run += __shfl(lane_incl, kWave - 1);
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
