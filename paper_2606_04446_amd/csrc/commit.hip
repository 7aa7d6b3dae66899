// Commit of the accepted path into the paged KV cache (sec. 3.3: a cycle
// consumes the verified cache and the previous bonus token; after joint
// verification the longest accepted prefix is committed and the prediction
// at the rejection point becomes the next anchor).
//
// Request b with context length C and accepted length L: the tree nodes at
// depths 0..L of the chosen path (the anchor, then the accepted drafts) have
// their K and V rows, computed in this pass, written at positions C..C+L of
// the request's pages, and the context length becomes C + L + 1. The bonus
// token is not written: the next cycle computes its K/V as the root of its
// tree. One workgroup per request moves 16-byte chunks; it is a pure copy
// (bytes in = bytes out).
#include "launchers.h"

namespace d2sd {

namespace {

constexpr int kCommitThreads = 256;

__global__ __launch_bounds__(kCommitThreads) void commit_kernel(
    int B, int hkv, int row_chunks, int num_pages, int max_pages, int max_ctx, const int* __restrict__ node_indptr,
    int total_nodes, const int* __restrict__ path_nodes, const int* __restrict__ accept_len,
    const uint4* __restrict__ k_tree, const uint4* __restrict__ v_tree, const int* __restrict__ page_table,
    int* __restrict__ ctx_len, uint4* __restrict__ k_cache, uint4* __restrict__ v_cache) {
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  const int C = clampi(ctx_len[b], 0, max_ctx);
  const int L = clampi(accept_len[b], 0, B - 1);
  const int base = clampi(node_indptr[b], 0, total_nodes);
  const int per_depth = hkv * row_chunks;          // 16-byte chunks of one token over all KV heads
  const int n = (L + 1) * per_depth;
  for (int i = t; i < n; i += kCommitThreads) {
    const int d = i / per_depth;
    const int rem = i - d * per_depth;
    const int h = rem / row_chunks;
    const int c = rem - h * row_chunks;
    const int local = path_nodes[(size_t)b * B + d];
    if (local < 0 || local >= total_nodes - base) continue;   // no overflow: base <= total_nodes
    const int node = base + local;
    const int pos = C + d;
    const int page = clampi(page_table[(size_t)b * max_pages + pos / D2SD_PAGE_SIZE], 0, num_pages - 1);
    const size_t dst = (((size_t)page * hkv + h) * D2SD_PAGE_SIZE + pos % D2SD_PAGE_SIZE) * row_chunks + c;
    const size_t src = ((size_t)node * hkv + h) * row_chunks + c;
    k_cache[dst] = k_tree[src];
    v_cache[dst] = v_tree[src];
  }
  __syncthreads();                                 // every thread has read ctx_len[b]
  if (t == 0) ctx_len[b] = C + L + 1;
}

}  // namespace

hipError_t launch_commit(int batch, int B, int hkv, int row_bytes, int num_pages, int max_pages, int max_ctx,
                         const int* node_indptr, int total_nodes, const int* path_nodes, const int* accept_len,
                         const void* k_tree, const void* v_tree, const int* page_table, int* ctx_len,
                         void* k_cache, void* v_cache, hipStream_t stream) {
  hipLaunchKernelGGL(commit_kernel, dim3(batch), dim3(kCommitThreads), 0, stream, B, hkv, row_bytes / 16,
                     num_pages, max_pages, max_ctx, node_indptr, total_nodes, path_nodes, accept_len,
                     static_cast<const uint4*>(k_tree), static_cast<const uint4*>(v_tree), page_table, ctx_len,
                     static_cast<uint4*>(k_cache), static_cast<uint4*>(v_cache));
  return hipGetLastError();
}

}  // namespace d2sd
