// Candidate-tree build (sec. 3.2 branch construction; sec. 3.3 (ii)-(iii)).
//
// One workgroup per request. The tree is produced in closed form: with the
// re-anchor positions sorted ascending and branch k (0-based rank) starting at
// node off_k = B + sum_{k' < k} (B - p_k'), the node n >= B of branch k sits at
// block position p_k + (n - off_k), and its ancestor-or-self set is the main
// prefix {0 .. p_k - 1} plus the branch run {off_k .. n}. A main node j sees
// {0 .. j}. Every mask word is therefore the union of two bit ranges, which is
// computed directly instead of walking parent pointers.
#include "launchers.h"

namespace d2sd {

namespace {

constexpr int kTreeThreads = 256;

__global__ __launch_bounds__(kTreeThreads) void tree_build_kernel(
    int B, int Kmax, const int* __restrict__ K, const int* __restrict__ p,
    const int* __restrict__ node_indptr, int total_nodes, int mask_words, int* __restrict__ parent,
    int* __restrict__ depth, int* __restrict__ path_id, uint32_t* __restrict__ anc_mask,
    int* __restrict__ path_leaf) {
  __shared__ int s_raw[D2SD_MAX_B];    // positions as given
  __shared__ int s_p[D2SD_MAX_B];      // positions sorted ascending
  __shared__ int s_off[D2SD_MAX_B + 1];
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  // All global inputs in one batch of independent loads: the row of p is
  // read whole (it is Kmax entries long whatever K[b] is), then ranked in LDS.
  const int Kb = clampi(K[b], 0, min(Kmax, B - 1));
  const int ip0 = node_indptr[b], ip1 = node_indptr[b + 1];
  if (t < min(Kmax, B - 1)) s_raw[t] = clampi(p[(size_t)b * Kmax + t], 1, B - 1);
  __syncthreads();

  // Rank sort: positions are distinct, so rank = number of smaller positions.
  if (t < Kb) {
    const int pt = s_raw[t];
    int rank = 0;
    for (int j = 0; j < Kb; ++j) {
      const int pj = s_raw[j];
      rank += (pj < pt) || (pj == pt && j < t);
    }
    s_p[rank] = pt;
  }
  __syncthreads();
  if (t == 0) {
    int off = B;
    for (int k = 0; k < Kb; ++k) {
      s_off[k] = off;
      off += B - s_p[k];
    }
    s_off[Kb] = off;
  }
  __syncthreads();

  const int base = clampi(ip0, 0, total_nodes);
  const int Nb = clampi(min(s_off[Kb], ip1 - base), 0, total_nodes - base);
  for (int n = t; n < Nb; n += kTreeThreads) {
    int pos, path, par, main_hi, br_lo, br_hi;
    if (n < B) {
      pos = n; path = 0; par = n - 1;
      main_hi = n + 1; br_lo = 0; br_hi = 0;
    } else {
      int k = 0;
      while (k + 1 < Kb && s_off[k + 1] <= n) ++k;
      const int pk = s_p[k];
      pos = pk + (n - s_off[k]);
      path = k + 1;
      par = (n == s_off[k]) ? pk - 1 : n - 1;
      main_hi = pk; br_lo = s_off[k]; br_hi = n + 1;
    }
    const size_t g = (size_t)base + n;
    parent[g] = par;
    depth[g] = pos;
    path_id[g] = path;
    uint32_t* row = anc_mask + g * mask_words;
    for (int w = 0; w < mask_words; ++w) row[w] = range_bits(0, main_hi, w) | range_bits(br_lo, br_hi, w);
  }
  for (int k = t; k <= Kmax; k += kTreeThreads) {
    int leaf = -1;
    if (k == 0) leaf = B - 1;
    else if (k <= Kb) leaf = s_off[k - 1] + (B - s_p[k - 1]) - 1;
    path_leaf[(size_t)b * (Kmax + 1) + k] = leaf;
  }
}

// Trees given as parent arrays (node 0 the root, parent[n] < n): the
// third-level cascade and resampled chains. Node n walks its parent links,
// setting one mask bit per ancestor-or-self and counting the depth; a parent
// outside [0, n) makes n a root of its own. path_id[n] counts the nodes m in
// 1..n whose parent is not m - 1 (path starts), by a chunked block scan.
__global__ __launch_bounds__(kTreeThreads) void tree_from_parents_kernel(
    const int* __restrict__ node_indptr, int total_nodes, int max_nodes, int mask_words,
    const int* __restrict__ parent, int* __restrict__ depth, int* __restrict__ path_id,
    uint32_t* __restrict__ anc_mask) {
  __shared__ int s_scan[kTreeThreads];
  __shared__ int s_carry;
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  const int base = clampi(node_indptr[b], 0, total_nodes);
  const int Nb = clampi(node_indptr[b + 1] - base, 0, min(max_nodes, total_nodes - base));
  auto par_of = [&](int n) {
    const int q = parent[base + n];
    return (q >= 0 && q < n) ? q : -1;
  };
  for (int n = t; n < Nb; n += kTreeThreads) {
    uint32_t* row = anc_mask + (size_t)(base + n) * mask_words;
    for (int w = 0; w < mask_words; ++w) row[w] = 0u;
    int d = -1;
    for (int a = n; a >= 0; a = par_of(a)) {
      row[a >> 5] |= 1u << (a & 31);
      ++d;
    }
    depth[base + n] = d;
  }
  if (t == 0) s_carry = 0;
  __syncthreads();
  for (int n0 = 0; n0 < Nb; n0 += kTreeThreads) {
    const int n = n0 + t;
    s_scan[t] = (n > 0 && n < Nb && parent[base + n] != n - 1) ? 1 : 0;
    __syncthreads();
    for (int dd = 1; dd < kTreeThreads; dd <<= 1) {
      const int v = t >= dd ? s_scan[t - dd] : 0;
      __syncthreads();
      s_scan[t] += v;
      __syncthreads();
    }
    const int carry = s_carry;
    if (n < Nb) path_id[base + n] = carry + s_scan[t];
    __syncthreads();
    if (t == kTreeThreads - 1) s_carry = carry + s_scan[t];
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_tree_from_parents(int batch, const int* node_indptr, int total_nodes, int max_nodes,
                                    int mask_words, const int* parent, int* depth, int* path_id,
                                    uint32_t* anc_mask, hipStream_t stream) {
  hipLaunchKernelGGL(tree_from_parents_kernel, dim3(batch), dim3(kTreeThreads), 0, stream, node_indptr,
                     total_nodes, max_nodes, mask_words, parent, depth, path_id, anc_mask);
  return hipGetLastError();
}

hipError_t launch_tree_build(int batch, int B, int Kmax, const int* K, const int* p,
                             const int* node_indptr, int total_nodes, int mask_words, int* parent,
                             int* depth, int* path_id, uint32_t* anc_mask, int* path_leaf,
                             hipStream_t stream) {
  hipLaunchKernelGGL(tree_build_kernel, dim3(batch), dim3(kTreeThreads), 0, stream, B, Kmax, K, p,
                     node_indptr, total_nodes, mask_words, parent, depth, path_id, anc_mask,
                     path_leaf);
  return hipGetLastError();
}

}  // namespace d2sd
