// Re-anchor selection on the device (sec. 3.1 Eq. 4, sec. 3.2 Eq. 5,
// sec. 3.3 (ii)) and the device node offsets of the candidate trees it
// produces, so that a verify step needs no host round-trip.
//
// r(i) = (c_1 c_2 ... c_i)(1 - c_{i+1}), i = 0..B-2, is the probability that
// exactly i drafts of the block are accepted when position k is accepted
// independently with probability c_k. It is evaluated in float64 with one
// fixed operation order (product from c_1 upward, then the factor 1 - c_{i+1},
// no contraction), so the selection is reproducible bit for bit. The K largest
// r(i) are kept, equal values going to the smaller i; prefix length i becomes
// the re-anchor block position p = i + 1.
#include "launchers.h"

namespace d2sd {

namespace {

constexpr int kSelectThreads = 64;    // one wave per request: B - 1 <= 63 prefix lengths
constexpr int kIndptrThreads = 256;

#pragma clang fp contract(off)
__device__ __attribute__((noinline)) double posterior(const float* c, int i) {
  double prod = 1.0;
  for (int k = 0; k < i; ++k) prod = prod * (double)c[k];
  return prod * (1.0 - (double)c[i]);
}

__global__ __launch_bounds__(kSelectThreads) void select_reanchor_kernel(
    int B, int Kmax, const float* __restrict__ conf, const int* __restrict__ K, int* __restrict__ p_out,
    double* __restrict__ r_out) {
  __shared__ double s_r[kSelectThreads];
  const int b = blockIdx.x;
  const int i = threadIdx.x;           // prefix length
  const int n = B - 1;                 // number of prefix lengths 0..B-2
  const float* c = conf + (size_t)b * n;
  const double r = i < n ? posterior(c, i) : 0.0;
  // Ranking key: a NaN posterior (from confidences outside [0, 1] or NaN)
  // ranks below every number, so the order stays total and exactly Kb
  // prefix lengths are kept.
  const double key = __builtin_isnan(r) ? -INFINITY : r;
  s_r[i] = key;
  __syncthreads();
  const int Kb = clampi(K[b], 0, min(Kmax, n));
  bool keep = false;
  if (i < n) {
    int rank = 0;                       // prefix lengths ordered before i
    for (int j = 0; j < n; ++j) {
      const double rj = s_r[j];
      rank += (rj > key) || (rj == key && j < i);
    }
    keep = rank < Kb;
    if (r_out) r_out[(size_t)b * n + i] = r;
  }
  // kept prefix lengths in ascending order: slot = kept lanes below this one
  const uint64_t kept = __ballot(keep);
  if (keep) {
    const int slot = __popcll(kept & ((1ull << i) - 1ull));
    if (slot < Kb) p_out[(size_t)b * Kmax + slot] = i + 1;
  }
  for (int k = Kb + i; k < Kmax; k += kSelectThreads) p_out[(size_t)b * Kmax + k] = -1;
}

// node_indptr[b+1] - node_indptr[b] = B + sum_k (B - p_k), with K and p
// clamped exactly as the tree builder clamps them.
__global__ __launch_bounds__(kIndptrThreads) void tree_indptr_kernel(int batch, int B, int Kmax,
                                                                     const int* __restrict__ K,
                                                                     const int* __restrict__ p,
                                                                     int* __restrict__ node_indptr) {
  __shared__ int s_scan[kIndptrThreads];
  __shared__ int s_carry;
  const int t = threadIdx.x;
  if (t == 0) {
    s_carry = 0;
    node_indptr[0] = 0;
  }
  __syncthreads();
  for (int b0 = 0; b0 < batch; b0 += kIndptrThreads) {
    const int b = b0 + t;
    int nb = 0;
    if (b < batch) {
      const int Kb = clampi(K[b], 0, min(Kmax, B - 1));
      nb = B;
      for (int k = 0; k < Kb; ++k) nb += B - clampi(p[(size_t)b * Kmax + k], 1, B - 1);
    }
    // inclusive scan of the chunk (Hillis-Steele)
    s_scan[t] = nb;
    __syncthreads();
    for (int d = 1; d < kIndptrThreads; d <<= 1) {
      const int v = t >= d ? s_scan[t - d] : 0;
      __syncthreads();
      s_scan[t] += v;
      __syncthreads();
    }
    const int carry = s_carry;
    if (b < batch) node_indptr[b + 1] = carry + s_scan[t];
    __syncthreads();
    if (t == kIndptrThreads - 1) s_carry = carry + s_scan[t];
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_select_reanchor(int batch, int B, int Kmax, const float* conf, const int* K, int* p_out,
                                  double* r_out, hipStream_t stream) {
  hipLaunchKernelGGL(select_reanchor_kernel, dim3(batch), dim3(kSelectThreads), 0, stream, B, Kmax, conf, K,
                     p_out, r_out);
  return hipGetLastError();
}

hipError_t launch_tree_indptr(int batch, int B, int Kmax, const int* K, const int* p, int* node_indptr,
                              hipStream_t stream) {
  hipLaunchKernelGGL(tree_indptr_kernel, dim3(1), dim3(kIndptrThreads), 0, stream, batch, B, Kmax, K, p,
                     node_indptr);
  return hipGetLastError();
}

}  // namespace d2sd
