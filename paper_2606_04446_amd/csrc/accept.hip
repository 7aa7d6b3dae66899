// Greedy longest-accepted-path selection and bonus token (sec. 2 "DFlash"
// prefix matching; sec. 3.3 (iv) longest accepted prefix across branches).
//
// One workgroup per request. Acceptance of a node is the AND of the match
// flags on its root path. It is computed for all nodes at once by pointer
// jumping (a parallel prefix scan along parent links): after round r every
// node holds the AND over its nearest 2^r path nodes and a pointer to its
// 2^r-th ancestor, so ceil(log2(B)) rounds cover any root path. The accepted
// length and the chosen node come from one max-reduction over the key
// (depth, -index), which implements "deepest accepted node, lowest canonical
// index on ties".
//
// The kernel is latency-bound (a few hundred nodes per request): every global
// input of a node is read in one batch of independent loads at the start and
// staged in LDS, so the match flags, the scan and the walk up the chosen path
// never wait on global memory again.
#include "launchers.h"

namespace d2sd {

namespace {

constexpr int kAcceptThreads = 256;
constexpr int kMaxNodes = D2SD_MAX_B + D2SD_MAX_B * (D2SD_MAX_B - 1) / 2;  // 2080

__global__ __launch_bounds__(kAcceptThreads) void accept_path_kernel(
    int B, const int* __restrict__ node_indptr, int total_nodes, const int* __restrict__ parent,
    const int* __restrict__ depth, const int* __restrict__ path_id, const int* __restrict__ draft,
    const int* __restrict__ argmax, int* __restrict__ accept_len, int* __restrict__ best_path,
    int* __restrict__ accept_node, int* __restrict__ path_nodes, int* __restrict__ out_tokens) {
  __shared__ uint8_t s_ok[2][kMaxNodes];
  __shared__ short s_up[2][kMaxNodes];
  __shared__ short s_par[kMaxNodes];
  __shared__ uint8_t s_dep[kMaxNodes];
  __shared__ int s_tok[kMaxNodes];
  __shared__ int s_arg[kMaxNodes];
  __shared__ int s_pid[kMaxNodes];
  __shared__ int s_pn[D2SD_MAX_B];
  __shared__ int s_tk[D2SD_MAX_B];
  __shared__ int s_best[kAcceptThreads / kWave];

  const int b = blockIdx.x;
  const int t = threadIdx.x;
  const int base = clampi(node_indptr[b], 0, total_nodes);
  const int Nb = clampi(node_indptr[b + 1] - base, 0, min(kMaxNodes, total_nodes - base));

  for (int c = t; c < Nb; c += kAcceptThreads) {
    int par = parent[base + c];
    if (par < 0 || par >= c) par = -1;   // canonical order puts parents first
    s_par[c] = (short)par;
    s_tok[c] = draft[base + c];
    s_arg[c] = argmax[base + c];
    s_pid[c] = path_id[base + c];
    s_dep[c] = (uint8_t)clampi(depth[base + c], 0, B - 1);
  }
  if (t < B) {
    s_pn[t] = -1;
    s_tk[t] = -1;
  }
  __syncthreads();
  for (int c = t; c < Nb; c += kAcceptThreads) {
    const short par = s_par[c];
    s_ok[0][c] = par < 0 || s_tok[c] == s_arg[par];
    s_up[0][c] = par;
  }
  __syncthreads();
  int cur = 0;
  for (int span = 1; span < B; span *= 2) {
    for (int c = t; c < Nb; c += kAcceptThreads) {
      uint8_t ok = s_ok[cur][c];
      short up = s_up[cur][c];
      if (up >= 0) {
        ok &= s_ok[cur][up];
        up = s_up[cur][up];
      }
      s_ok[cur ^ 1][c] = ok;
      s_up[cur ^ 1][c] = up;
    }
    __syncthreads();
    cur ^= 1;
  }

  // key = depth * 65536 + (65535 - index) over accepted nodes; the root is
  // always accepted, so the maximum exists whenever Nb > 0.
  int best = -1;
  for (int c = t; c < Nb; c += kAcceptThreads)
    if (s_ok[cur][c]) best = max(best, (int)s_dep[c] * 65536 + (65535 - c));
  for (int off = kWave / 2; off > 0; off /= 2) best = max(best, __shfl_xor(best, off));
  if ((t % kWave) == 0) s_best[t / kWave] = best;
  __syncthreads();

  if (t == 0) {
    for (int w = 1; w < kAcceptThreads / kWave; ++w) best = max(best, s_best[w]);
    if (best < 0) {
      accept_len[b] = 0; best_path[b] = 0; accept_node[b] = -1;
    } else {
      const int L = best / 65536;
      const int chosen = 65535 - best % 65536;
      accept_len[b] = L;
      best_path[b] = s_pid[chosen];
      accept_node[b] = chosen;
      // Walk up from the chosen node; depth L sits at slot L.
      int c = chosen;
      for (int d = L; d >= 0 && c >= 0; --d) {
        s_pn[d] = c;
        if (d >= 1) s_tk[d - 1] = s_tok[c];
        c = s_par[c];
      }
      s_tk[L] = s_arg[chosen];
    }
  }
  __syncthreads();
  if (t < B) {
    path_nodes[(size_t)b * B + t] = s_pn[t];
    out_tokens[(size_t)b * B + t] = s_tk[t];
  }
}

}  // namespace

hipError_t launch_accept_path(int batch, int B, const int* node_indptr, int total_nodes,
                              const int* parent, const int* depth, const int* path_id,
                              const int* draft, const int* argmax, int* accept_len, int* best_path,
                              int* accept_node, int* path_nodes, int* out_tokens,
                              hipStream_t stream) {
  hipLaunchKernelGGL(accept_path_kernel, dim3(batch), dim3(kAcceptThreads), 0, stream, B,
                     node_indptr, total_nodes, parent, depth, path_id, draft, argmax, accept_len,
                     best_path, accept_node, path_nodes, out_tokens);
  return hipGetLastError();
}

}  // namespace d2sd
