// Launchers of the tree, selection, accept and commit kernels (implemented in
// their .hip files); the C ABI in api.hip validates arguments first. The
// attention launchers are declared in common.h next to the attention plan.
#pragma once

#include "common.h"

namespace d2sd {

hipError_t launch_tree_build(int batch, int B, int Kmax, const int* K, const int* p,
                             const int* node_indptr, int total_nodes, int mask_words, int* parent,
                             int* depth, int* path_id, uint32_t* anc_mask, int* path_leaf,
                             hipStream_t stream);

hipError_t launch_tree_from_parents(int batch, const int* node_indptr, int total_nodes, int max_nodes,
                                    int mask_words, const int* parent, int* depth, int* path_id,
                                    uint32_t* anc_mask, hipStream_t stream);

hipError_t launch_select_reanchor(int batch, int B, int Kmax, const float* conf, const int* K, int* p_out,
                                  double* r_out, hipStream_t stream);

hipError_t launch_tree_indptr(int batch, int B, int Kmax, const int* K, const int* p, int* node_indptr,
                              hipStream_t stream);

hipError_t launch_commit(int batch, int B, int hkv, int row_bytes, int num_pages, int max_pages, int max_ctx,
                         const int* node_indptr, int total_nodes, const int* path_nodes, const int* accept_len,
                         const void* k_tree, const void* v_tree, const int* page_table, int* ctx_len,
                         void* k_cache, void* v_cache, hipStream_t stream);

hipError_t launch_accept_path(int batch, int B, const int* node_indptr, int total_nodes,
                              const int* parent, const int* depth, const int* path_id,
                              const int* draft, const int* argmax, int* accept_len, int* best_path,
                              int* accept_node, int* path_nodes, int* out_tokens,
                              hipStream_t stream);

hipError_t launch_sample_targets(int batch, const int* node_indptr, int total_nodes, int max_nodes,
                                 const int* parent, const int* draft, int vocab, int dtype, const void* logits,
                                 float temperature, const float* uniform, int* context_rep, int* tokens,
                                 hipStream_t stream);

}  // namespace d2sd
