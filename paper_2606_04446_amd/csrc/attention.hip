// Cascade verify attention over the candidate tree (sec. 3.3 (iv): the K+1
// candidates are verified in one target pass with shared-prefix cascade
// attention; sec. 1, contribution 2: the shared context is reused instead of
// being replicated per candidate).
//
// Work decomposition. For one request b and KV head h, the M = N_b * G query
// rows (tree node n, query head h*G+g, row index n*G+g) all attend to the same
// context keys, so they are stacked into the column dimension of one dense
// contraction. A work item is (request, KV head, row group, context split); a
// row group is 128 rows, four waves of one 32-row column tile each. Every
// 32-key K/V tile of the split is fetched from HBM once per row group, staged
// in an LDS ring of two stages and consumed by all rows of the group. The tree
// keys of the request are appended to split 0 under the ancestor mask, so the
// tree state joins the context state through the same online log-sum-exp
// rescale.
//
// Per tile and wave: S^T = K Q^T with MFMA (keys on the MFMA row axis,
// queries on the column axis), so a lane owns one query and 16 keys of each
// 32-key block; the row max needs one cross-half exchange and the row sum
// stays lane-local. P^T leaves the accumulator already in MFMA B-operand
// order, and O^T += V^T P^T takes the V^T fragments in the matching key order
// (bf16: transposing LDS reads of the row-major V tile; fp32: per-element
// reads of the key-major tile). Split partials (O divided by its row sum, in
// the input dtype; running max in log2 units and running sum in fp32) go to
// the workspace and a second kernel merges them by log-sum-exp; a request with
// a single split is finalised in place.
//
// The fp32 kernel stages tiles through registers. The bf16 kernel copies them
// by LDS DMA, in one of three workgroup shapes (three waves per SIMD in each):
// 4 waves of 32 query rows, three workgroups per CU; 12 waves sharing one K/V
// ring, one workgroup per CU; or 12 waves over the sequence of all streams'
// query tiles (the packed kernel). It moves the running max (and rescales O
// and l) only when it grows by more than 2^8, and skips masking on interior
// context tiles.
#include <math.h>

#include <mutex>

#include "common.h"

namespace d2sd {

namespace {

constexpr int kD = 128;
constexpr int kThreads = 256;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct Params {
  const void* q;
  const void* k_cache;
  const void* v_cache;
  const int* page_table;
  const int* ctx_len;
  const void* k_tree;
  const void* v_tree;
  const int* node_indptr;
  const uint32_t* anc_mask;
  void* out;
  float* lse;
  void* ws_o;   // [n_ch_max, total_rows, D] split outputs normalised by their row sum, in the input dtype
  float* ws_m;  // [n_ch_max, total_rows]
  float* ws_l;  // [n_ch_max, total_rows]
  int batch, hq, hkv, G, stage;
  int total_nodes, max_nodes, max_ctx, num_pages, max_pages, mask_words;
  int split, n_ch_max, n_rg_max, items;
  float c2;  // sm_scale * log2(e)
};

// Tiling of the generic kernel (instantiated for fp32; bf16 has its own kernel).
template <typename T>
struct Tile;

template <>
struct Tile<float> {
  static constexpr int KT = 32;
  static constexpr int WT = 1;
  static constexpr int KS = 130;        // K row stride (floats)
  static constexpr int VS = 136;        // V row stride (floats), V kept key-major
  static constexpr int K_ELEMS = KT * KS;
  static constexpr int V_ELEMS = KT * VS;
};

__device__ __forceinline__ f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma(float a, float b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint4 zero4() { return make_uint4(0u, 0u, 0u, 0u); }

// s_waitcnt vmcnt(0): wait for every outstanding vector-memory access of the
// wave (gfx9 encoding: vmcnt 0, expcnt and lgkmcnt left at their maxima).
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0f70); }

// Pointer to the first element of key `kabs` of request b / KV head h, or null
// when the key lies outside [0, key_end). Context keys go through the page
// table, tree keys index the tree K/V rows of the request.
template <typename T>
__device__ __forceinline__ const T* key_row(const Params& p, const T* base_cache, const T* base_tree,
                                            bool tree, int b, int h, int node_base, int kabs,
                                            int key_end) {
  if (kabs >= key_end) return nullptr;
  if (tree) return base_tree + ((size_t)(node_base + kabs) * p.hkv + h) * kD;
  int page = p.page_table[(size_t)b * p.max_pages + (kabs >> 4)];
  page = clampi(page, 0, p.num_pages - 1);
  return base_cache + (((size_t)page * p.hkv + h) * D2SD_PAGE_SIZE + (kabs & 15)) * kD;
}

// ---- staging of one K/V tile: global -> registers -> LDS ------------------

struct StageF32 {
  uint4 k[4];
  uint4 v[4];
};

// fp32: 32 keys x 128 dims per tile; chunk c = t + 256 i covers key c/32,
// dims (c%32)*4..+4, for K and V alike (V stays key-major).
__device__ __forceinline__ void load_tile(const Params& p, StageF32& st, bool tree, int b, int h,
                                          int node_base, int key0, int key_end) {
  const float* kc = static_cast<const float*>(p.k_cache);
  const float* vc = static_cast<const float*>(p.v_cache);
  const float* kt = static_cast<const float*>(p.k_tree);
  const float* vt = static_cast<const float*>(p.v_tree);
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int key = 8 * i + (t >> 5);
    const int d4 = (t & 31) * 4;
    const float* rk = key_row(p, kc, kt, tree, b, h, node_base, key0 + key, key_end);
    const float* rv = key_row(p, vc, vt, tree, b, h, node_base, key0 + key, key_end);
    st.k[i] = rk ? *reinterpret_cast<const uint4*>(rk + d4) : zero4();
    st.v[i] = rv ? *reinterpret_cast<const uint4*>(rv + d4) : zero4();
  }
}

__device__ __forceinline__ void store_tile(const StageF32& st, float* sK, float* sV) {
  using C = Tile<float>;
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int key = 8 * i + (t >> 5);
    const int d4 = (t & 31) * 4;
    *reinterpret_cast<uint2*>(sK + key * C::KS + d4) = make_uint2(st.k[i].x, st.k[i].y);
    *reinterpret_cast<uint2*>(sK + key * C::KS + d4 + 2) = make_uint2(st.k[i].z, st.k[i].w);
    *reinterpret_cast<uint4*>(sV + key * C::VS + d4) = st.v[i];
  }
}

template <typename T>
struct Frag;
template <>
struct Frag<float> {
  using Q = float;
  static constexpr int QN = 64;  // k-steps over the head dim (2 dims each)
};

// Head-dim assignment of the S^T = K Q^T k-steps (must agree for K and Q).
// bf16: step s, lane half hf holds dims hf*64 + s*8 .. +8.
// fp32: step s, lane half hf holds dim 2s + hf.
__device__ __forceinline__ void load_q(const Params& p, bf16x8 (&qf)[8], const __bf16* row, int hf) {
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    if (row) {
      uint4 u = *reinterpret_cast<const uint4*>(row + hf * 64 + s * 8);
      qf[s] = __builtin_bit_cast(bf16x8, u);
    } else {
      qf[s] = __builtin_bit_cast(bf16x8, zero4());
    }
  }
}
__device__ __forceinline__ void load_q(const Params& p, float (&qf)[64], const float* row, int hf) {
#pragma unroll
  for (int s = 0; s < 64; ++s) qf[s] = row ? row[2 * s + hf] : 0.0f;
}

// S^T block (32 keys starting at key row kb of the LDS tile) for one query tile.
__device__ __forceinline__ f32x16 score_block(const float* sK, int kb, const float (&qf)[64],
                                              int lane) {
  using C = Tile<float>;
  f32x16 acc = {};
  const int hf = lane >> 5;
  const float* base = sK + (kb + (lane & 31)) * C::KS + hf;
#pragma unroll
  for (int s = 0; s < 64; ++s) acc = mfma(base[2 * s], qf[s], acc);
  return acc;
}

// O^T (4 dim tiles of 32) += V^T P^T for one 32-key block of the tile.
// fp32: accumulator slot i of lane half hf is key kb + (i/4)*8 + hf*4 + i%4.
__device__ __forceinline__ void pv_block(const float* sV, int kb, const f32x16& pr, f32x16 (&o)[4],
                                         int lane) {
  using C = Tile<float>;
  const int hf = lane >> 5;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int key = kb + (i >> 2) * 8 + hf * 4 + (i & 3);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) o[dt] = mfma(sV[key * C::VS + dt * 32 + (lane & 31)], pr[i], o[dt]);
  }
}

template <typename T>
struct Stage;
template <>
struct Stage<float> {
  using type = StageF32;
};

template <typename T>
__device__ __forceinline__ void store_out(T* dst, const float* v4);
template <>
__device__ __forceinline__ void store_out<__bf16>(__bf16* dst, const float* v) {
  __bf16 h[4] = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
  *reinterpret_cast<uint2*>(dst) = *reinterpret_cast<const uint2*>(h);
}
template <>
__device__ __forceinline__ void store_out<float>(float* dst, const float* v) {
  *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
}

// kNode: the non-cascade baseline, one workgroup per (request, node, KV
// head) streaming the whole context for that node's query heads.
template <typename T, bool kNode>
__device__ __forceinline__ void attention_body(const Params& p) {
  using C = Tile<T>;
  using QF = typename Frag<T>::Q;
  constexpr int KT = C::KT;
  constexpr int QN = Frag<T>::QN;
  constexpr int NBLK = KT / 32;   // 32-key blocks per tile
  constexpr int WT = C::WT;
  constexpr int GROUP_ROWS = 4 * WT * kRowsPerTile;

  __shared__ __attribute__((aligned(16))) T smem[2 * (C::K_ELEMS + C::V_ELEMS)];

  // ---- work item (XCD-aware: consecutive items share an XCD and its L2) ----
  const int per_xcd = gridDim.x / 8;
  const int item = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (item >= p.items) return;
  int rest = item;
  int rg = 0, ch = 0, n_sel = 0;
  if (kNode) {
    n_sel = rest % p.max_nodes; rest /= p.max_nodes;
  } else {
    rg = rest % p.n_rg_max; rest /= p.n_rg_max;
    ch = rest % p.n_ch_max; rest /= p.n_ch_max;
  }
  const int h = rest % p.hkv;
  const int b = rest / p.hkv;

  const int node_base = clampi(p.node_indptr[b], 0, p.total_nodes);
  const int Nb = clampi(p.node_indptr[b + 1] - node_base, 0, min(p.max_nodes, p.total_nodes - node_base));
  const int Mb = Nb * p.G;
  // rows [r_lo, r_hi) of the (request, KV head) column block owned by this workgroup
  int r_lo, r_hi;
  if (kNode) {
    if (n_sel >= Nb) return;
    r_lo = n_sel * p.G;
    r_hi = r_lo + p.G;
  } else {
    r_lo = rg * GROUP_ROWS;
    if (r_lo >= Mb) return;
    r_hi = min(Mb, r_lo + GROUP_ROWS);
  }
  const int Cb = clampi(p.ctx_len[b], 0, p.max_ctx);
  const bool use_ctx = p.stage != D2SD_STAGE_TREE;
  const bool use_tree = p.stage != D2SD_STAGE_PREFIX;
  const int n_ch_b = use_ctx ? max(1, ceil_div(Cb, p.split)) : 1;
  if (ch >= n_ch_b) return;
  const int c0 = use_ctx ? ch * p.split : 0;
  const int c1 = use_ctx ? min(Cb, c0 + p.split) : 0;
  const int n_ctx_tiles = c1 > c0 ? ceil_div(c1 - c0, KT) : 0;
  const int n_tree_tiles = (use_tree && ch == 0) ? ceil_div(Nb, KT) : 0;
  const int n_tiles = n_ctx_tiles + n_tree_tiles;

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int hf = lane >> 5;
  const int tiles_wg = ceil_div(r_hi - r_lo, kRowsPerTile);
  // query tiles of this wave: wave and wave + 4 (balanced over the 4 SIMDs)
  const int nq = min(WT, (wave < tiles_wg) + (wave + 4 < tiles_wg));

  QF qf[WT][QN];
  int qnode[WT];
  int qrow[WT];  // global output row (node * hq + head) or -1
#pragma unroll
  for (int j = 0; j < WT; ++j) {
    const int r = r_lo + (wave + 4 * j) * kRowsPerTile + (lane & 31);
    const bool valid = j < nq && r < r_hi;
    const int n = valid ? r / p.G : 0;
    const int g = valid ? r % p.G : 0;
    qnode[j] = n;
    qrow[j] = valid ? (node_base + n) * p.hq + h * p.G + g : -1;
    const T* row = valid ? static_cast<const T*>(p.q) + (size_t)qrow[j] * kD : nullptr;
    load_q(p, qf[j], row, hf);
  }

  f32x16 o[WT][4];
  float m_run[WT], l_run[WT];
#pragma unroll
  for (int j = 0; j < WT; ++j) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) o[j][dt] = f32x16{};
    m_run[j] = -INFINITY;
    l_run[j] = 0.0f;
  }

  // two LDS stages, each [K tile | V tile]
  auto stage_k = [&](int i) { return smem + i * (C::K_ELEMS + C::V_ELEMS); };
  auto stage_v = [&](int i) { return smem + i * (C::K_ELEMS + C::V_ELEMS) + C::K_ELEMS; };
  typename Stage<T>::type st;

  auto tile_src = [&](int j, bool& tree, int& key0, int& key_end) {
    tree = j >= n_ctx_tiles;
    key0 = tree ? (j - n_ctx_tiles) * KT : c0 + j * KT;
    key_end = tree ? Nb : c1;
  };

  if (n_tiles > 0) {
    bool tr; int k0, ke;
    tile_src(0, tr, k0, ke);
    load_tile(p, st, tr, b, h, node_base, k0, ke);
    store_tile(st, stage_k(0), stage_v(0));
  }
  __syncthreads();

  for (int jt = 0; jt < n_tiles; ++jt) {
    const int cur = jt & 1;
    if (jt + 1 < n_tiles) {
      bool tr; int k0, ke;
      tile_src(jt + 1, tr, k0, ke);
      load_tile(p, st, tr, b, h, node_base, k0, ke);
    }
    bool is_tree; int key0, key_end;
    tile_src(jt, is_tree, key0, key_end);
#pragma unroll
    for (int j = 0; j < WT; ++j) {
      if (j >= nq) break;
      // scores of this tile: NBLK blocks of 32 keys, slot i of block kb is key
      // key0 + 32 kb + (i/4)*8 + hf*4 + i%4
      f32x16 s[NBLK];
#pragma unroll
      for (int kb = 0; kb < NBLK; ++kb) s[kb] = score_block(stage_k(cur), 32 * kb, qf[j], lane);
      uint64_t vis = ~0ull;  // visible-key bits of this tile for the lane's node
      if (is_tree) {
        const uint32_t* mrow = p.anc_mask + (size_t)(node_base + qnode[j]) * p.mask_words;
        const int w0 = key0 >> 5;
        const uint32_t lo = w0 < p.mask_words ? mrow[w0] : 0u;
        const uint32_t hi = (KT > 32 && w0 + 1 < p.mask_words) ? mrow[w0 + 1] : 0u;
        vis = (uint64_t)lo | ((uint64_t)hi << 32);
      }
      const int nvalid = key_end - key0;  // keys >= nvalid are padding
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < NBLK; ++kb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int k = 32 * kb + (i >> 2) * 8 + hf * 4 + (i & 3);
          const bool ok = k < nvalid && ((vis >> k) & 1ull);
          s[kb][i] = ok ? s[kb][i] : -INFINITY;
          mx = fmaxf(mx, s[kb][i]);
        }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[j], mx);
      const float m_use = m_new == -INFINITY ? 0.0f : m_new;
      const float alpha = __builtin_amdgcn_exp2f((m_run[j] - m_use) * p.c2);
      const float moff = m_use * p.c2;
      float lsum = 0.0f;
#pragma unroll
      for (int kb = 0; kb < NBLK; ++kb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float e = __builtin_amdgcn_exp2f(fmaf(s[kb][i], p.c2, -moff));
          s[kb][i] = e;
          lsum += e;
        }
      }
      l_run[j] = l_run[j] * alpha + lsum;
      m_run[j] = m_new;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) o[j][dt] *= alpha;
#pragma unroll
      for (int kb = 0; kb < NBLK; ++kb) pv_block(stage_v(cur), 32 * kb, s[kb], o[j], lane);
    }
    if (jt + 1 < n_tiles) store_tile(st, stage_k(cur ^ 1), stage_v(cur ^ 1));
    __syncthreads();
  }

  // ---- epilogue: finalise (single split) or write the split partial ----
  const bool direct = n_ch_b == 1;
#pragma unroll
  for (int j = 0; j < WT; ++j) {
    if (j >= nq) break;
    const float l_all = l_run[j] + __shfl_xor(l_run[j], 32);
    if (qrow[j] < 0) continue;
    const size_t row = (size_t)qrow[j];
    if (direct) {
      const float inv = l_all > 0.0f ? 1.0f / l_all : 0.0f;
      T* dst = static_cast<T*>(p.out) + row * kD;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          float v[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] = o[j][dt][q4 * 4 + r] * inv;
          store_out<T>(dst + dt * 32 + q4 * 8 + hf * 4, v);
        }
      }
      if (p.lse && hf == 0)
        p.lse[row] = l_all > 0.0f ? (m_run[j] * p.c2 + __log2f(l_all)) * kLn2 : -INFINITY;
    } else {
      const size_t prow = (size_t)ch * ((size_t)p.total_nodes * p.hq) + row;
      const float inv = l_all > 0.0f ? 1.0f / l_all : 0.0f;
      T* dst = static_cast<T*>(p.ws_o) + prow * kD;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          float v[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] = o[j][dt][q4 * 4 + r] * inv;
          store_out<T>(dst + dt * 32 + q4 * 8 + hf * 4, v);
        }
      }
      if (hf == 0) {
        p.ws_m[prow] = l_all > 0.0f ? m_run[j] * p.c2 : -INFINITY;
        p.ws_l[prow] = l_all;
      }
    }
  }
}

template <typename T>
__global__ __launch_bounds__(kThreads) void cascade_attention_kernel(Params p) {
  attention_body<T, false>(p);
}
template <typename T>
__global__ __launch_bounds__(kThreads) void noncascade_attention_kernel(Params p) {
  attention_body<T, true>(p);
}

// ---------------------------------------------------------------------------
// bf16 kernel (the hot path), in two workgroup shapes with the same body and
// one 32-query column tile per wave (163 VGPRs: three waves per SIMD):
//  - 4 waves (128 query rows), three workgroups per CU (40 KB of LDS each):
//    every SIMD interleaves three independent waves;
//  - 12 waves (384 query rows), one workgroup per CU: the three waves of a
//    SIMD share one K/V ring, so a context split is copied from HBM once per
//    384 rows instead of once per 128 (eight of the waves issue the copies).
// The host planner takes the wide shape when its rows fill the waves as well. K/V tiles of 32 keys are
// copied global -> LDS by the LDS DMA path (global_load_lds_dwordx4: no
// staging registers, no VALU) into a two-stage ring: the copy of tile j+1 is
// in flight while tile j is consumed. Both tiles keep the natural [key][dim]
// layout with 16-byte chunks XOR-swizzled by row:
//   K: chunk c of row r sits at c ^ (r & 15)   (b128 A-operand reads of 16
//      consecutive keys hit 16 distinct bank groups)
//   V: chunk c of row r sits at c ^ 4(r & 3)   (transposing b64 reads)
// V^T fragments for O^T += V^T P^T come from ds_read_b64_tr_b16: in each
// 16-lane group, lane i points at V[k0 + i/4][d0 + 4(i%4)] and receives keys
// k0..k0+3 of dim d0 + i, which is the key order of the P^T slots.

namespace bf {
constexpr int MAX_SPLIT_PAGES = 2048;    // page ids of one context split staged in LDS
constexpr int KT = 32;                   // keys per tile (a 40 KB workgroup: three per CU)
constexpr int NKB = KT / 32;             // 32-key MFMA blocks per tile
constexpr int ROW_BYTES = kD * 2;        // 256 B per key row
constexpr int TILE_BYTES = KT * ROW_BYTES;  // 8 KB for K (and for V)
constexpr int BLOCKS = KT / 4;           // 1 KB (four-row) DMA blocks per K or V tile
constexpr float kRescaleLog2 = 8.0f;     // move the running max when it grows by > 2^8
// Workgroup shape: W waves, the first COPY_WAVES of which issue the copies,
// WAVE_BLOCKS K (and V) blocks each.
template <int W>
struct Shape {
  static constexpr int WAVES = W;
  static constexpr int THREADS = W * kWave;
  static constexpr int COPY_WAVES = W < 8 ? W : 8;
  static constexpr int WAVE_BLOCKS = BLOCKS / COPY_WAVES;
  static_assert(BLOCKS % COPY_WAVES == 0, "copy blocks per wave");
};
}  // namespace bf

typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 lds_b128(const char* base, int off) {
  return *reinterpret_cast<const uint4*>(base + off);
}
__device__ __forceinline__ s16x4 lds_tr16(const char* base, int off) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(base + off));
}
// LDS DMA copies are issued as inline asm so that the compiler does not
// track them: its own tracking cannot tell ring stages apart and would make
// every later LDS read wait for all copies in flight (vmcnt(0)). The kernel
// orders copies and reads itself (sync_keep); untracked loads can only
// lengthen the compiler's own vmcnt waits, never shorten them. The s_nop
// covers the M0-write to LDS-DMA hazard. Each lane's 16 bytes land at
// M0 + 16 * lane.
__device__ __forceinline__ uint32_t lds_addr(const char* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)p;
}
__device__ __forceinline__ void dma16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ void dma16s(const char* base, uint32_t lane_off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(lane_off), "s"(base), "s"(lds)
               : "memory", "m0");
}

// s_waitcnt vmcnt(n) lgkmcnt(0) then s_barrier; the asm statement is also a
// compiler memory barrier. Waves keep up to n of their own LDS DMAs in flight.
template <int N>
__device__ __forceinline__ void sync_keep() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  // gfx9 s_waitcnt: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] at [15:14]
  __builtin_amdgcn_s_waitcnt((N & 15) | 0x0070 | ((N >> 4) << 14));
  asm volatile("s_barrier" ::: "memory");
}
struct TileSrc {
  bool tree;
  int key0;
  int key_end;
};

// Per-lane constants of the DMA copy: copying wave w (w < CW) copies K/V
// blocks w, w + CW, ... (rows 4b .. 4b+3 of the tile, one 16-byte chunk per lane).
template <int CW>
struct DmaLane {
  static constexpr int N = bf::BLOCKS / CW;
  int row[N];   // tile row of the lane's chunk in each block
  int kcol[N];  // element offset of the logical K chunk to fetch
  int vcol[N];  // element offset of the logical V chunk to fetch
};

template <int CW>
__device__ __forceinline__ DmaLane<CW> dma_lane(int wave, int lane) {
  DmaLane<CW> d;
#pragma unroll
  for (int j = 0; j < DmaLane<CW>::N; ++j) {
    const int blk = wave + CW * j;
    const int r = 4 * blk + (lane >> 4);
    const int p = lane & 15;          // physical chunk written by this lane
    d.row[j] = r;
    d.kcol[j] = (p ^ (r & 15)) * 8;
    d.vcol[j] = (p ^ ((r & 3) << 2)) * 8;
  }
  return d;
}

// Issue the LDS DMA of one K/V tile into a stage (sK, sV: 16 KB each).
// Rows past the valid keys are copied from row 0 (their scores are masked,
// so they only need to be finite).
template <int CW>
__device__ __forceinline__ void dma_tile(const Params& p, const TileSrc& ts, int h, int node_base,
                                         const int* s_pid, int c0, const DmaLane<CW>& d, char* sK, char* sV) {
  const __bf16* kc = static_cast<const __bf16*>(p.k_cache);
  const __bf16* vc = static_cast<const __bf16*>(p.v_cache);
  const int nvalid = ts.key_end - ts.key0;
  const int wave = threadIdx.x >> 6;
#pragma unroll
  for (int j = 0; j < DmaLane<CW>::N; ++j) {
    const int r = d.row[j];
    const int rs = r < nvalid ? r : 0;
    size_t rowoff;
    const __bf16* kb;
    const __bf16* vb;
    if (!ts.tree) {
      const int key = ts.key0 + rs;
      const int ph = s_pid[(key - c0) >> 4];
      rowoff = ((size_t)ph * D2SD_PAGE_SIZE + (key & 15)) * kD;
      kb = kc;
      vb = vc;
    } else {
      rowoff = ((size_t)(node_base + ts.key0 + rs) * p.hkv + h) * kD;
      kb = static_cast<const __bf16*>(p.k_tree);
      vb = static_cast<const __bf16*>(p.v_tree);
    }
    const uint32_t blk_off = (uint32_t)__builtin_amdgcn_readfirstlane(wave + CW * j) * 1024u;
    dma16(kb + rowoff + d.kcol[j], lds_addr(sK) + blk_off);
    dma16(vb + rowoff + d.vcol[j], lds_addr(sV) + blk_off);
  }
}
// Fast copy of a full context tile. A four-row block lies in one page (tiles
// start on page boundaries), so its source is a wave-uniform page base plus a
// per-lane offset that depends only on the lane and the block's row within
// the page, which is the same for every block of a wave. The copy takes the
// staged page ids (page * hkv + h) of the wave's blocks, read beforehand by
// ctx_tile_pages, so that the steady state can read them a step ahead.
constexpr int kPagesPerTile = bf::KT / D2SD_PAGE_SIZE;
template <int CW>
__device__ __forceinline__ void ctx_tile_pages(const int* s_pid, int tile, int wave_s, int (&ph)[bf::BLOCKS / CW]) {
#pragma unroll
  for (int j = 0; j < bf::BLOCKS / CW; ++j) ph[j] = s_pid[kPagesPerTile * tile + ((wave_s + CW * j) >> 2)];
}
template <int CW>
__device__ __forceinline__ void dma_ctx_pages(const Params& p, const int (&ph)[bf::BLOCKS / CW], int wave_s,
                                              uint32_t koff, uint32_t voff, const char* sK, const char* sV) {
  const char* kc = static_cast<const char*>(p.k_cache);
  const char* vc = static_cast<const char*>(p.v_cache);
#pragma unroll
  for (int j = 0; j < bf::BLOCKS / CW; ++j) {
    const uint32_t blk = wave_s + CW * j;
    const size_t off = (size_t)(uint32_t)__builtin_amdgcn_readfirstlane(ph[j]) << 12;  // 16 rows x 256 B
    dma16s(kc + off, koff, lds_addr(sK) + blk * 1024u);
    dma16s(vc + off, voff, lds_addr(sV) + blk * 1024u);
  }
}

// Per-lane LDS read offsets (bytes from the stage base).
struct ReadLane {
  int k[8];   // K A-operand chunk of k-step st for key row lane%32 (block 0)
  int v[4];   // V transposing read for dim tile dt (first 4 keys of k-step 0)
};

__device__ __forceinline__ ReadLane read_lane(int lane) {
  ReadLane rl;
  const int hf = lane >> 5;
  const int kr = lane & 31;
#pragma unroll
  for (int st = 0; st < 8; ++st) rl.k[st] = kr * bf::ROW_BYTES + (((hf * 8 + st) ^ (kr & 15)) << 4);
  const int grp = lane >> 4;          // 16-lane group: dims (grp&1)*16.., keys +4*(grp>>1)
  const int i = lane & 15;
  const int row = 4 * (grp >> 1) + (i >> 2);
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
    const int c = dt * 4 + (grp & 1) * 2 + ((i & 3) >> 1);       // logical 16-byte chunk
    rl.v[dt] = row * bf::ROW_BYTES + ((c ^ ((row & 3) << 2)) << 4) + ((i & 1) << 3);
  }
  return rl;
}

// S^T of one query tile for a key tile (NKB blocks of 32 keys).
__device__ __forceinline__ void qk_tile(const char* sK, const ReadLane& rl, const bf16x8 (&q)[8],
                                        f32x16 (&s)[bf::NKB]) {
#pragma unroll
  for (int kb = 0; kb < bf::NKB; ++kb) s[kb] = f32x16{};
#pragma unroll
  for (int st = 0; st < 8; ++st) {
#pragma unroll
    for (int kb = 0; kb < bf::NKB; ++kb) {
      const bf16x8 a = __builtin_bit_cast(bf16x8, lds_b128(sK, rl.k[st] + kb * 32 * bf::ROW_BYTES));
      s[kb] = mfma(a, q[st], s[kb]);
    }
  }
}

// O^T += V^T P^T over a key tile (2 NKB k-steps of 16 keys).
__device__ __forceinline__ void pv_tile(const char* sV, const ReadLane& rl, const bf16x8 (&pf)[2 * bf::NKB],
                                        f32x16 (&o)[4]) {
#pragma unroll
  for (int ks = 0; ks < 2 * bf::NKB; ++ks) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const s16x4 lo = lds_tr16(sV, rl.v[dt] + (ks * 16) * bf::ROW_BYTES);
      const s16x4 hi = lds_tr16(sV, rl.v[dt] + (ks * 16 + 8) * bf::ROW_BYTES);
      typedef short s16x8 __attribute__((ext_vector_type(8)));
      const s16x8 a8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      o[dt] = mfma(__builtin_bit_cast(bf16x8, a8), pf[ks], o[dt]);
    }
  }
}

__device__ __forceinline__ float xhalf_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Mask keys of a partial or tree tile: slot i of block kb is key
// 32 kb + (i/4)*8 + hf*4 + i%4 of the tile. `vis` holds the visible keys of
// the tile; after shifting out the lane half's offset every slot tests a
// fixed bit.
__device__ __forceinline__ void mask_tile(f32x16 (&s)[bf::NKB], int nvalid, uint64_t vis, int hf) {
  const uint64_t in_range = nvalid >= 64 ? ~0ull : ((1ull << max(nvalid, 0)) - 1ull);
  const uint64_t m = (vis & in_range) >> (hf * 4);
  const uint32_t w[2] = {(uint32_t)m, (uint32_t)(m >> 32)};
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int bit = (i >> 2) * 8 + (i & 3);
#pragma unroll
    for (int kb = 0; kb < bf::NKB; ++kb) s[kb][i] = ((w[kb] >> bit) & 1u) ? s[kb][i] : -INFINITY;
  }
}

// Online softmax of one query tile over a key tile: updates the running max /
// sum / output scale and leaves bf16 probabilities in B-operand order.
__device__ __forceinline__ void softmax_tile(f32x16 (&s)[bf::NKB], float& m_run, float& l_run, f32x16 (&o)[4],
                                             bf16x8 (&pf)[2 * bf::NKB], float c2) {
  float mx = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < bf::NKB; ++kb)
#pragma unroll
    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[kb][i]);
  mx = xhalf_max(mx);
  const float m_new = fmaxf(m_run, mx);
  const bool grow = (m_new - m_run) * c2 > bf::kRescaleLog2;  // false when both are -inf
  if (__ballot(grow)) {
    const float alpha = m_run == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f((m_run - m_new) * c2);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) o[dt] *= alpha;
    l_run *= alpha;
    m_run = m_new;
  }
  const float moff = m_run == -INFINITY ? 0.0f : m_run * c2;
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  float la = 0.0f, lb = 0.0f;
#pragma unroll
  for (int kb = 0; kb < bf::NKB; ++kb) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      bf16x8 v;
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = (__bf16)__builtin_amdgcn_exp2f(fmaf(s[kb][8 * t + j], c2, -moff));
#pragma unroll
      for (int j = 0; j < 8; j += 4) {
        la = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v[j], v[j + 1]}, ones, la, false);
        lb = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v[j + 2], v[j + 3]}, ones, lb, false);
      }
      pf[2 * kb + t] = v;
    }
  }
  l_run += la + lb;
}

// Visible-key bits of a tree tile for the node of a query row.
__device__ __forceinline__ uint64_t tree_bits(const Params& p, int node_base, int node, int key0) {
  const uint32_t* mrow = p.anc_mask + (size_t)(node_base + node) * p.mask_words;
  const int w0 = key0 >> 5;
  const uint32_t lo = w0 < p.mask_words ? mrow[w0] : 0u;
  const uint32_t hi = w0 + 1 < p.mask_words ? mrow[w0 + 1] : 0u;
  return (uint64_t)lo | ((uint64_t)hi << 32);
}

template <bool kNode, int W>
__device__ __forceinline__ void bf16_attention_body(const Params& p) {
  using S = bf::Shape<W>;
  constexpr int CW = S::COPY_WAVES;
  constexpr int GROUP_ROWS = S::WAVES * kRowsPerTile;
  // the two stages of the K/V ring
  __shared__ __attribute__((aligned(1024))) char sk0[bf::TILE_BYTES], sv0[bf::TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char sk1[bf::TILE_BYTES], sv1[bf::TILE_BYTES];
  __shared__ __attribute__((aligned(16))) int s_pid[bf::MAX_SPLIT_PAGES + 4];

  // ---- work item (XCD-aware: consecutive items share an XCD and its L2) ----
  const int per_xcd = gridDim.x / 8;
  const int item = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (item >= p.items) return;
  int rest = item;
  int rg = 0, ch = 0, n_sel = 0;
  if (kNode) {
    n_sel = rest % p.max_nodes; rest /= p.max_nodes;
  } else {
    rg = rest % p.n_rg_max; rest /= p.n_rg_max;
    ch = rest % p.n_ch_max; rest /= p.n_ch_max;
  }
  const int h = rest % p.hkv;
  const int b = rest / p.hkv;
  const int node_base = clampi(p.node_indptr[b], 0, p.total_nodes);
  const int Nb = clampi(p.node_indptr[b + 1] - node_base, 0, min(p.max_nodes, p.total_nodes - node_base));
  const int Mb = Nb * p.G;
  int r_lo, r_hi;
  if (kNode) {
    if (n_sel >= Nb) return;
    r_lo = n_sel * p.G;
    r_hi = r_lo + p.G;
  } else {
    r_lo = rg * GROUP_ROWS;
    if (r_lo >= Mb) return;
    r_hi = min(Mb, r_lo + GROUP_ROWS);
  }
  const int Cb = clampi(p.ctx_len[b], 0, p.max_ctx);
  const bool use_ctx = p.stage != D2SD_STAGE_TREE;
  const bool use_tree = p.stage != D2SD_STAGE_PREFIX;
  const int n_ch_b = use_ctx ? max(1, ceil_div(Cb, p.split)) : 1;
  if (ch >= n_ch_b) return;
  const int c0 = use_ctx ? ch * p.split : 0;
  const int c1 = use_ctx ? min(Cb, c0 + p.split) : 0;
  const int n_ctx_tiles = c1 > c0 ? ceil_div(c1 - c0, bf::KT) : 0;
  const int n_tree_tiles = (use_tree && ch == 0) ? ceil_div(Nb, bf::KT) : 0;
  const int n_tiles = n_ctx_tiles + n_tree_tiles;

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int hf = lane >> 5;
  const int r = r_lo + wave * kRowsPerTile + (lane & 31);
  const bool active = r_lo + wave * kRowsPerTile < r_hi;   // wave owns at least one row
  const bool valid = r < r_hi;
  const int qnode = valid ? r / p.G : 0;
  const int qrow = valid ? (node_base + qnode) * p.hq + h * p.G + r % p.G : -1;

  // page ids of this split (the split length is capped so they fit)
  {
    const int npg = ceil_div(c1 - c0, D2SD_PAGE_SIZE);
    const int* pt = p.page_table + (size_t)b * p.max_pages + (c0 >> 4);
    for (int i = threadIdx.x; i < npg; i += S::THREADS) s_pid[i] = clampi(pt[i], 0, p.num_pages - 1) * p.hkv + h;
  }
  bf16x8 q[8];
  load_q(p, q, valid ? static_cast<const __bf16*>(p.q) + (size_t)qrow * kD : nullptr, hf);
  f32x16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x16{};
  float m_run = -INFINITY, l_run = 0.0f;
  // Retire the Q loads on every path before the first copy is queued: the
  // compiler's later waits for them would otherwise also wait for the copies.
  wait_vmem();
  __syncthreads();

  auto src = [&](int j) {
    TileSrc ts;
    ts.tree = j >= n_ctx_tiles;
    ts.key0 = ts.tree ? (j - n_ctx_tiles) * bf::KT : c0 + j * bf::KT;
    ts.key_end = ts.tree ? Nb : c1;
    return ts;
  };
  const DmaLane<CW> dl = dma_lane<CW>(wave, lane);
  const ReadLane rl = read_lane(lane);
  // fast-path lane offsets: row within the page and swizzled source chunk
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const int prow = 4 * (wave & 3) + (lane >> 4);
  const uint32_t koff = prow * bf::ROW_BYTES + (((lane & 15) ^ prow) << 4);
  const uint32_t voff = prow * bf::ROW_BYTES + (((lane & 15) ^ ((prow & 3) << 2)) << 4);
  auto copy_tile = [&](int j, const char* sK, const char* sV) {
    if (wave_s >= CW) return;   // wave-uniform: only the copying waves
    const TileSrc ts = src(j);
    if (!ts.tree && ts.key_end - ts.key0 >= bf::KT) {
      int ph[S::WAVE_BLOCKS];
      ctx_tile_pages<CW>(s_pid, j, wave_s, ph);
      dma_ctx_pages<CW>(p, ph, wave_s, koff, voff, sK, sV);
    } else
      dma_tile<CW>(p, ts, h, node_base, s_pid, c0, dl, const_cast<char*>(sK), const_cast<char*>(sV));
  };

  // prologue: tile 0 in flight
  if (n_tiles > 0) copy_tile(0, sk0, sv0);

  // One tile: wait for its copy and for every wave to be done with the
  // previous tile, queue the next tile into the stage that one used, compute.
  auto step = [&](int jt, const char* cK, const char* cV, char* nK, char* nV) {
    sync_keep<0>();
    if (jt + 1 < n_tiles) copy_tile(jt + 1, nK, nV);
    if (!active) return;
    const TileSrc ts = src(jt);
    const int nvalid = ts.key_end - ts.key0;
    f32x16 s[bf::NKB];
    qk_tile(cK, rl, q, s);
    if (ts.tree || nvalid < bf::KT) {
      uint64_t vis = ~0ull;
      if (ts.tree) {
        vis = tree_bits(p, node_base, qnode, ts.key0);  // waits for in-flight copies too (tree tiles are few)
      }
      mask_tile(s, nvalid, vis, hf);
    }
    bf16x8 pf[2 * bf::NKB];
    softmax_tile(s, m_run, l_run, o, pf, p.c2);
    pv_tile(cV, rl, pf, o);
  };
  // Steady state: the tile consumed and the tile queued are both whole
  // context tiles, so the step needs no masking, no choice of copy path, and
  // reads the page ids of the tile it will queue next one step ahead (the
  // staged page list does not change after the prologue).
  const int n_full = c1 > c0 ? (c1 - c0) / bf::KT : 0;
  int ph_next[S::WAVE_BLOCKS];
  if (n_full > 2 && wave_s < CW) ctx_tile_pages<CW>(s_pid, 1, wave_s, ph_next);
  auto fast_step = [&](int jt, const char* cK, const char* cV, const char* nK, const char* nV) {
    sync_keep<0>();
    if (wave_s < CW) {
      dma_ctx_pages<CW>(p, ph_next, wave_s, koff, voff, nK, nV);    // tile jt + 1
      if (jt + 2 < n_full) ctx_tile_pages<CW>(s_pid, jt + 2, wave_s, ph_next);
    }
    if (!active) return;
    f32x16 s[bf::NKB];
    qk_tile(cK, rl, q, s);
    bf16x8 pf[2 * bf::NKB];
    softmax_tile(s, m_run, l_run, o, pf, p.c2);
    pv_tile(cV, rl, pf, o);
  };
  int jt = 0;
  for (; jt + 2 < n_full; jt += 2) {   // both steps queue a whole context tile
    fast_step(jt, sk0, sv0, sk1, sv1);
    fast_step(jt + 1, sk1, sv1, sk0, sv0);
  }
  for (; jt < n_tiles; jt += 2) {      // the rest: partial and tree tiles (stage parity kept)
    step(jt, sk0, sv0, sk1, sv1);
    if (jt + 1 < n_tiles) step(jt + 1, sk1, sv1, sk0, sv0);
  }

  // ---- epilogue: finalise (single split) or write the split partial ----
  if (!active) return;
  const float l_all = l_run + __shfl_xor(l_run, 32);
  if (!valid) return;
  const size_t row = (size_t)qrow;
  if (n_ch_b == 1) {
    const float inv = l_all > 0.0f ? 1.0f / l_all : 0.0f;
    __bf16* dst = static_cast<__bf16*>(p.out) + row * kD;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        float v[4];
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) v[rr] = o[dt][q4 * 4 + rr] * inv;
        store_out<__bf16>(dst + dt * 32 + q4 * 8 + hf * 4, v);
      }
    }
    if (p.lse && hf == 0) p.lse[row] = l_all > 0.0f ? (m_run * p.c2 + __log2f(l_all)) * kLn2 : -INFINITY;
  } else {
    const size_t prow = (size_t)ch * ((size_t)p.total_nodes * p.hq) + row;
    const float inv = l_all > 0.0f ? 1.0f / l_all : 0.0f;
    __bf16* dst = static_cast<__bf16*>(p.ws_o) + prow * kD;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        float v[4];
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) v[rr] = o[dt][q4 * 4 + rr] * inv;
        store_out<__bf16>(dst + dt * 32 + q4 * 8 + hf * 4, v);
      }
    }
    if (hf == 0) {
      p.ws_m[prow] = l_all > 0.0f ? m_run * p.c2 : -INFINITY;
      p.ws_l[prow] = l_all;
    }
  }
}

// ---------------------------------------------------------------------------
// Packed twelve-wave bf16 kernel. The query tiles of all streams (request b,
// KV head h, context split ch: T_b = ceil(N_b G / 32) tiles of 32 rows each,
// n_ch_max splits per request, the splits a request does not need are empty)
// form one sequence in (b, h, ch, tile) order; workgroup i takes tiles
// 12 i .. 12 i + 11, one per wave. Consecutive waves on the same stream form
// a segment that shares one K/V ring, so no wave is idle for lack of rows
// and a stream is read by the one to three workgroups that hold its tiles
// (neighbours in the dispatch order, on one XCD). The host takes this shape
// only when every stream has at least pk::MIN_TILES tiles, so that a
// workgroup holds at most pk::SEGS segments. All twelve waves share the
// copies: segment s's tile is eight 1 KB K/V block pairs, pair 8 s + j goes
// to wave (8 s + j) mod 12.
namespace pk {
constexpr int WAVES = 12;
constexpr int THREADS = WAVES * kWave;
constexpr int SEGS = 3;
constexpr int MIN_TILES = kPackedMinTiles;            // 12 consecutive tiles span <= 3 streams
constexpr int MAX_SPLIT_PAGES = kPackedMaxSplit / D2SD_PAGE_SIZE;
constexpr int MAX_BATCH = kPackedMaxBatch;
static_assert(WAVES / MIN_TILES + 1 <= SEGS, "segments per workgroup");
constexpr int SEG_BYTES = 4 * bf::TILE_BYTES;   // two stages x (K, V)
constexpr int PAIRS = 2;                // block pairs per wave and round: waves w and w + 12 of 24
}  // namespace pk

struct PackedSeg {
  int b, h, ch, node_base, Nb, c0, c1, n_ctx_tiles, n_tiles, n_full, n_ch_b;
};

__device__ __forceinline__ int wave_incl_scan(int x, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  return x;
}

// Tiles of request b over all its streams.
__device__ __forceinline__ int request_tiles(const Params& p, int b) {
  const int nb0 = clampi(p.node_indptr[b], 0, p.total_nodes);
  const int Nb = clampi(p.node_indptr[b + 1] - nb0, 0, min(p.max_nodes, p.total_nodes - nb0));
  return ceil_div(Nb * p.G, kRowsPerTile) * p.hkv * p.n_ch_max;
}

__device__ void bf16_packed_body(const Params& p) {
  __shared__ __attribute__((aligned(1024))) char ring[pk::SEGS * pk::SEG_BYTES];
  __shared__ __attribute__((aligned(16))) int s_pid[pk::SEGS][pk::MAX_SPLIT_PAGES];
  __shared__ int s_pref[pk::MAX_BATCH + 1];
  __shared__ int s_wsum[pk::WAVES];
  __shared__ int s_gs[pk::WAVES];
  __shared__ PackedSeg s_seg[pk::SEGS];

  const int per_xcd = gridDim.x / 8;
  const int item = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int hf = lane >> 5;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const int batch = min(p.batch, pk::MAX_BATCH);

  // ---- tiles before each request (block scan; up to 3 requests per thread) ----
  {
    constexpr int PER = (pk::MAX_BATCH + pk::THREADS - 1) / pk::THREADS;
    int loc[PER];
    int sum = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int b = tid * PER + k;
      loc[k] = sum;
      sum += b < batch ? request_tiles(p, b) : 0;
    }
    const int incl = wave_incl_scan(sum, lane);
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    int off = 0;
    for (int w = 0; w < wave; ++w) off += s_wsum[w];
    const int excl = off + incl - sum;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int b = tid * PER + k;
      if (b < batch) s_pref[b] = excl + loc[k];
    }
    if (tid == 0) {
      int tot = 0;
      for (int w = 0; w < pk::WAVES; ++w) tot += s_wsum[w];
      s_pref[batch] = tot;
    }
    __syncthreads();
  }

  // ---- this wave's tile: stream (b, h, ch) and tile index ti within it ----
  const int t = item * pk::WAVES + wave_s;
  int gs = -1, ti = 0, wb = 0;
  if (t < s_pref[batch]) {
    int lo = 0, hi = batch;                 // largest b with s_pref[b] <= t
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (s_pref[mid] <= t) lo = mid; else hi = mid;
    }
    wb = lo;
    const int per_stream = (s_pref[wb + 1] - s_pref[wb]) / (p.hkv * p.n_ch_max);   // T_b
    const int local = t - s_pref[wb];
    const int sidx = per_stream > 0 ? local / per_stream : 0;
    ti = per_stream > 0 ? local - sidx * per_stream : 0;
    gs = wb * p.hkv * p.n_ch_max + sidx;    // (b, h, ch) in sequence order
  }
  if (lane == 0) s_gs[wave_s] = gs;
  __syncthreads();
  // segment of this wave: count of stream starts among waves 0..wave
  int seg = -1, nseg = 0;
  for (int w = 0; w < pk::WAVES; ++w) {
    const bool start = s_gs[w] >= 0 && (w == 0 || s_gs[w] != s_gs[w - 1]);
    nseg += start;
    if (w == wave_s) seg = s_gs[w] >= 0 ? nseg - 1 : -1;
  }
  nseg = min(nseg, pk::SEGS);
  if (seg >= pk::SEGS) seg = -1;            // not reached when the host's size rule holds
  const bool seg_leader = seg >= 0 && (wave_s == 0 || s_gs[wave_s - 1] != gs);
  if (seg_leader && lane == 0) {
    PackedSeg g;
    const int sidx = gs - wb * p.hkv * p.n_ch_max;
    g.b = wb;
    g.h = sidx / p.n_ch_max;
    g.ch = sidx - g.h * p.n_ch_max;
    g.node_base = clampi(p.node_indptr[wb], 0, p.total_nodes);
    g.Nb = clampi(p.node_indptr[wb + 1] - g.node_base, 0, min(p.max_nodes, p.total_nodes - g.node_base));
    const int Cb = clampi(p.ctx_len[wb], 0, p.max_ctx);
    const bool use_ctx = p.stage != D2SD_STAGE_TREE;
    const bool use_tree = p.stage != D2SD_STAGE_PREFIX;
    g.n_ch_b = use_ctx ? max(1, ceil_div(Cb, p.split)) : 1;
    g.c0 = use_ctx ? g.ch * p.split : 0;
    g.c1 = use_ctx ? min(Cb, g.c0 + p.split) : 0;
    if (g.ch >= g.n_ch_b) g.c1 = g.c0;      // an empty stream
    g.n_ctx_tiles = g.c1 > g.c0 ? ceil_div(g.c1 - g.c0, bf::KT) : 0;
    const int n_tree = (use_tree && g.ch == 0) ? ceil_div(g.Nb, bf::KT) : 0;
    g.n_tiles = g.ch < g.n_ch_b ? g.n_ctx_tiles + n_tree : 0;
    g.n_full = g.c1 > g.c0 ? (g.c1 - g.c0) / bf::KT : 0;
    s_seg[seg] = g;
  }
  __syncthreads();

  // ---- page ids of every segment's split ----
  for (int sg = 0; sg < nseg; ++sg) {
    const PackedSeg& g = s_seg[sg];
    const int npg = min(ceil_div(g.c1 - g.c0, D2SD_PAGE_SIZE), pk::MAX_SPLIT_PAGES);
    const int* pt = p.page_table + (size_t)g.b * p.max_pages + (g.c0 >> 4);
    for (int i = tid; i < npg; i += pk::THREADS) s_pid[sg][i] = clampi(pt[i], 0, p.num_pages - 1) * p.hkv + g.h;
  }

  // ---- this wave's rows ----
  auto uni = [](int x) { return __builtin_amdgcn_readfirstlane(x); };
  PackedSeg my{};
  if (seg >= 0) {
    const PackedSeg g = s_seg[seg];
    my.b = uni(g.b); my.h = uni(g.h); my.ch = uni(g.ch); my.node_base = uni(g.node_base); my.Nb = uni(g.Nb);
    my.c0 = uni(g.c0); my.c1 = uni(g.c1); my.n_ctx_tiles = uni(g.n_ctx_tiles); my.n_tiles = uni(g.n_tiles);
    my.n_full = uni(g.n_full); my.n_ch_b = uni(g.n_ch_b);
  }
  const int Mb = my.Nb * p.G;
  const int r_lo = ti * kRowsPerTile;
  // a wave of an existing stream writes its rows even with no tile to
  // attend to (an empty context in the prefix stage: O = 0, lse = -inf)
  const bool active = seg >= 0 && my.ch < my.n_ch_b && r_lo < Mb;
  const int r = r_lo + (lane & 31);
  const bool valid = active && r < Mb;
  const int qnode = valid ? r / p.G : 0;
  const int qrow = valid ? (my.node_base + qnode) * p.hq + my.h * p.G + r % p.G : -1;
  bf16x8 q[8];
  load_q(p, q, valid ? static_cast<const __bf16*>(p.q) + (size_t)qrow * kD : nullptr, hf);
  f32x16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x16{};
  float m_run = -INFINITY, l_run = 0.0f;
  wait_vmem();          // every global load retired before the first (untracked) copy
  __syncthreads();

  int n_rounds = 0, n_fast = 1 << 30;
  for (int sg = 0; sg < nseg; ++sg) {
    n_rounds = max(n_rounds, s_seg[sg].n_tiles);
    if (s_seg[sg].n_tiles > 0) n_fast = min(n_fast, s_seg[sg].n_full - 1);
  }
  n_rounds = uni(n_rounds);
  n_fast = uni(max(0, min(n_fast, n_rounds)));

  // LDS read offsets within this wave's segment ring
  ReadLane rl = read_lane(lane);
  {
    const int so = max(seg, 0) * pk::SEG_BYTES;
#pragma unroll
    for (int i = 0; i < 8; ++i) rl.k[i] += so;
#pragma unroll
    for (int i = 0; i < 4; ++i) rl.v[i] += so;
  }
  // Copy pairs of this wave: pair pr = wave + 12 jj (jj < PAIRS) when pr < 8 nseg;
  // pair pr is segment pr / 8, block pr % 8 (tile rows 4 blk .. 4 blk + 3), and
  // blk % 4 = wave % 4 for both pairs, so the fast-path lane offsets are per wave.
  const int prow = 4 * (wave_s & 3) + (lane >> 4);
  const uint32_t koff = prow * bf::ROW_BYTES + (((lane & 15) ^ prow) << 4);
  const uint32_t voff = prow * bf::ROW_BYTES + (((lane & 15) ^ ((prow & 3) << 2)) << 4);
  const char* kc = static_cast<const char*>(p.k_cache);
  const char* vc = static_cast<const char*>(p.v_cache);
  const uint32_t ring_lds = lds_addr(ring);
  int pr_sg[pk::PAIRS], pr_blk[pk::PAIRS], pr_tiles[pk::PAIRS];
#pragma unroll
  for (int jj = 0; jj < pk::PAIRS; ++jj) {
    const int pr = wave_s + pk::WAVES * jj;
    pr_sg[jj] = pr >> 3;
    pr_blk[jj] = pr & 7;
    pr_tiles[jj] = pr < 8 * nseg ? uni(s_seg[pr >> 3].n_tiles) : 0;   // 0: no such pair
  }
  // page ids of the fast copies of tile j (read one round ahead)
  auto dst_of = [&](int jj, int stage) {
    return ring_lds + pr_sg[jj] * pk::SEG_BYTES + stage * (2 * bf::TILE_BYTES) + pr_blk[jj] * 1024u;
  };
  // copy of tile j of the pairs' segments, any tile kind
  auto copy_any = [&](int j, int stage) {
#pragma unroll
    for (int jj = 0; jj < pk::PAIRS; ++jj) {
      if (j >= pr_tiles[jj]) continue;
      const PackedSeg& g = s_seg[pr_sg[jj]];
      const uint32_t dst = dst_of(jj, stage);
      const int n_ctx = uni(g.n_ctx_tiles);
      const bool tree = j >= n_ctx;
      const int c0 = uni(g.c0);
      const int key0 = tree ? (j - n_ctx) * bf::KT : c0 + j * bf::KT;
      const int nvalid = (tree ? uni(g.Nb) : uni(g.c1)) - key0;
      const int rr = 4 * pr_blk[jj] + (lane >> 4);
      const int rs = rr < nvalid ? rr : 0;
      const int pc = lane & 15;
      size_t rowoff;
      const __bf16* kb;
      const __bf16* vb;
      if (!tree) {
        const int key = key0 + rs;
        rowoff = ((size_t)s_pid[pr_sg[jj]][min((key - c0) >> 4, pk::MAX_SPLIT_PAGES - 1)] * D2SD_PAGE_SIZE +
                  (key & 15)) * kD;
        kb = static_cast<const __bf16*>(p.k_cache);
        vb = static_cast<const __bf16*>(p.v_cache);
      } else {
        rowoff = ((size_t)(uni(g.node_base) + key0 + rs) * p.hkv + uni(g.h)) * kD;
        kb = static_cast<const __bf16*>(p.k_tree);
        vb = static_cast<const __bf16*>(p.v_tree);
      }
      dma16(kb + rowoff + (pc ^ (rr & 15)) * 8, dst);
      dma16(vb + rowoff + (pc ^ ((rr & 3) << 2)) * 8, dst + bf::TILE_BYTES);
    }
  };
  const char* ringc = ring;
  auto compute = [&](int j, int stage, bool fast) {
    if (!active || j >= my.n_tiles) return;
    const char* sK = ringc + stage * (2 * bf::TILE_BYTES);
    const char* sV = sK + bf::TILE_BYTES;
    f32x16 sc[bf::NKB];
    qk_tile(sK, rl, q, sc);
    if (!fast) {
      const bool tree = j >= my.n_ctx_tiles;
      const int key0 = tree ? (j - my.n_ctx_tiles) * bf::KT : my.c0 + j * bf::KT;
      const int nvalid = (tree ? my.Nb : my.c1) - key0;
      if (tree || nvalid < bf::KT) {
        const uint64_t vis = tree ? tree_bits(p, my.node_base, qnode, key0) : ~0ull;
        mask_tile(sc, nvalid, vis, hf);
      }
    }
    bf16x8 pf[2 * bf::NKB];
    softmax_tile(sc, m_run, l_run, o, pf, p.c2);
    pv_tile(sV, rl, pf, o);
  };

  // prologue: tile 0 of every segment in flight
  if (n_rounds > 0) copy_any(0, 0);
  // Steady state: rounds j < n_fast consume, and queue, whole context tiles
  // of every live segment (n_fast <= n_full - 1 <= n_tiles - 1), so a round
  // needs no tile checks and no masks; the page ids of the copy after next
  // are read a round ahead.
  bool pr_on[pk::PAIRS];
#pragma unroll
  for (int jj = 0; jj < pk::PAIRS; ++jj) pr_on[jj] = pr_tiles[jj] > 0;
  const bool computes = active && my.n_tiles > 0;
  auto steady_copy = [&](int jt, int stage, const int (&ph)[pk::PAIRS]) {
#pragma unroll
    for (int jj = 0; jj < pk::PAIRS; ++jj) {
      if (!pr_on[jj]) continue;
      const size_t off = (size_t)(uint32_t)uni(ph[jj]) << 12;    // 16 rows x 256 B
      const uint32_t dst = dst_of(jj, stage);
      dma16s(kc + off, koff, dst);
      dma16s(vc + off, voff, dst + bf::TILE_BYTES);
    }
  };
  auto steady_pages = [&](int jt, int (&ph)[pk::PAIRS]) {
#pragma unroll
    for (int jj = 0; jj < pk::PAIRS; ++jj)
      if (pr_on[jj]) ph[jj] = s_pid[pr_sg[jj]][min(2 * jt + (pr_blk[jj] >> 2), pk::MAX_SPLIT_PAGES - 1)];
  };
  auto steady_compute = [&](int stage) {
    if (!computes) return;
    const char* sK = ringc + stage * (2 * bf::TILE_BYTES);
    f32x16 sc[bf::NKB];
    qk_tile(sK, rl, q, sc);
    bf16x8 pf[2 * bf::NKB];
    softmax_tile(sc, m_run, l_run, o, pf, p.c2);
    pv_tile(sK + bf::TILE_BYTES, rl, pf, o);
  };
  int ph_next[pk::PAIRS] = {0, 0};
  if (n_fast > 1) steady_pages(1, ph_next);
  int j = 0;
  for (; j + 1 < n_fast; j += 2) {
    sync_keep<0>();
    steady_copy(j + 1, 1, ph_next);      // j + 1 < n_fast
    steady_pages(j + 2, ph_next);
    steady_compute(0);
    sync_keep<0>();
    steady_copy(j + 2, 0, ph_next);      // j + 2 <= n_fast: still a whole context tile of every live segment
    steady_pages(j + 3, ph_next);
    steady_compute(1);
  }
  // the rest: partial and tree tiles (stage j % 2)
  for (; j < n_rounds; ++j) {
    sync_keep<0>();
    if (j + 1 < n_rounds) copy_any(j + 1, (j + 1) & 1);
    compute(j, j & 1, j < n_fast);
  }

  // ---- epilogue: finalise (single split) or write the split partial ----
  if (!active) return;
  const float l_all = l_run + __shfl_xor(l_run, 32);
  if (!valid) return;
  const size_t row = (size_t)qrow;
  if (my.n_ch_b == 1) {
    const float inv = l_all > 0.0f ? 1.0f / l_all : 0.0f;
    __bf16* dst = static_cast<__bf16*>(p.out) + row * kD;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        float v[4];
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) v[rr] = o[dt][q4 * 4 + rr] * inv;
        store_out<__bf16>(dst + dt * 32 + q4 * 8 + hf * 4, v);
      }
    }
    if (p.lse && hf == 0) p.lse[row] = l_all > 0.0f ? (m_run * p.c2 + __log2f(l_all)) * kLn2 : -INFINITY;
  } else {
    const size_t prow2 = (size_t)my.ch * ((size_t)p.total_nodes * p.hq) + row;
    const float inv = l_all > 0.0f ? 1.0f / l_all : 0.0f;
    __bf16* dst = static_cast<__bf16*>(p.ws_o) + prow2 * kD;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        float v[4];
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) v[rr] = o[dt][q4 * 4 + rr] * inv;
        store_out<__bf16>(dst + dt * 32 + q4 * 8 + hf * 4, v);
      }
    }
    if (hf == 0) {
      p.ws_m[prow2] = l_all > 0.0f ? m_run * p.c2 : -INFINITY;
      p.ws_l[prow2] = l_all;
    }
  }
}

__global__ __launch_bounds__(pk::THREADS) __attribute__((amdgpu_waves_per_eu(3)))
void cascade_bf16_packed_kernel(Params p) {
  bf16_packed_body(p);
}

__global__ __launch_bounds__(bf::Shape<kBf16Waves>::THREADS) __attribute__((amdgpu_waves_per_eu(3)))
void cascade_bf16_kernel(Params p) {
  bf16_attention_body<false, kBf16Waves>(p);
}
__global__ __launch_bounds__(bf::Shape<kBf16WideWaves>::THREADS) __attribute__((amdgpu_waves_per_eu(3)))
void cascade_bf16_wide_kernel(Params p) {
  bf16_attention_body<false, kBf16WideWaves>(p);
}
// The non-cascade baseline: the same body, one workgroup per (request, node, KV head).
__global__ __launch_bounds__(bf::Shape<kBf16Waves>::THREADS) __attribute__((amdgpu_waves_per_eu(3)))
void noncascade_bf16_kernel(Params p) {
  bf16_attention_body<true, kBf16Waves>(p);
}

// Log-sum-exp reduction of the split partials of every output row (rows of
// single-split requests were finalised by the attention kernel). A row takes
// GROUPS groups of 16 threads (8 dims per thread); group g folds splits g,
// g + GROUPS, ... in one pass with a running max, so the loads of one split
// never wait on the values of another and the unrolled loop keeps several
// splits in flight; with several groups their states are then combined in
// group order through LDS. A workgroup takes merge_rows(GROUPS) consecutive
// rows of one request: the request comes from the grid, so a thread needs
// only the request's node range and context length before it reads the
// partials. Many splits (short contexts in small batches) take four groups,
// which shortens the chain per thread and gives small batches more
// workgroups.
struct MergeState {
  float m, l;
  float acc[8];
};

// Eight consecutive dims of a split's normalised output.
__device__ __forceinline__ void load_partial8(const float* src, float (&v)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(src);
  const float4 b = *reinterpret_cast<const float4*>(src + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void load_partial8(const __bf16* src, float (&v)[8]) {
  const uint4 u = *reinterpret_cast<const uint4*>(src);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

template <typename T, int GROUPS>
__global__ __launch_bounds__(kThreads) void split_merge_kernel(Params p, int chunks) {
  constexpr int ROWS = merge_rows(GROUPS);
  static_assert(ROWS * GROUPS * 16 == kThreads, "16 threads per group and row");
  __shared__ MergeState s_st[GROUPS > 1 ? kThreads : 1];
  const int b = blockIdx.x / chunks;
  const int chunk = blockIdx.x % chunks;
  const int node_base = clampi(p.node_indptr[b], 0, p.total_nodes);
  const int Nb = clampi(p.node_indptr[b + 1] - node_base, 0, min(p.max_nodes, p.total_nodes - node_base));
  const int Cb = clampi(p.ctx_len[b], 0, p.max_ctx);
  const int n_ch_b = max(1, ceil_div(Cb, p.split));
  const int rl = threadIdx.x / (16 * GROUPS);            // row within the workgroup
  const int g = (threadIdx.x / 16) % GROUPS;             // split group
  const int d0 = (threadIdx.x & 15) * 8;
  const int r = chunk * ROWS + rl;                        // row within the request
  const bool live = n_ch_b > 1 && r < Nb * p.hq;
  const int row = node_base * p.hq + r;
  const size_t stride = (size_t)p.total_nodes * p.hq;
  float M = -INFINITY, L = 0.0f;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (live) {
#pragma unroll 4
    for (int s = g; s < n_ch_b; s += GROUPS) {
      const size_t pr = s * stride + row;
      const float ms = p.ws_m[pr];
      const float ls = p.ws_l[pr];
      float v[8];
      load_partial8(static_cast<const T*>(p.ws_o) + pr * kD + d0, v);
      const float Mn = fmaxf(M, ms);
      if (Mn == -INFINITY) continue;                        // no keys so far
      const float a = __builtin_amdgcn_exp2f(M - Mn);       // 0 while M is -inf
      const float w = __builtin_amdgcn_exp2f(ms - Mn) * ls; // 0 for an empty split
      L = L * a + w;
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = acc[i] * a + w * v[i];
      M = Mn;
    }
  }
  if constexpr (GROUPS > 1) {
    MergeState& st = s_st[threadIdx.x];
    st.m = M;
    st.l = L;
#pragma unroll
    for (int i = 0; i < 8; ++i) st.acc[i] = acc[i];
    __syncthreads();
    if (g != 0) return;
#pragma unroll
    for (int gg = 1; gg < GROUPS; ++gg) {
      const MergeState& o = s_st[threadIdx.x + 16 * gg];
      const float Mn = fmaxf(M, o.m);
      if (Mn == -INFINITY) continue;
      const float a = __builtin_amdgcn_exp2f(M - Mn);
      const float w = __builtin_amdgcn_exp2f(o.m - Mn);
      L = L * a + w * o.l;
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = acc[i] * a + w * o.acc[i];
      M = Mn;
    }
  }
  if (!live) return;
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  float o[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = acc[i] * inv;
  T* dst = static_cast<T*>(p.out) + (size_t)row * kD + d0;
  store_out<T>(dst, o);
  store_out<T>(dst + 4, o + 4);
  if (p.lse && (threadIdx.x & 15) == 0) p.lse[row] = L > 0.0f ? (M + __log2f(L)) * kLn2 : -INFINITY;
}

// The cascade merge as a standalone operator: merge two normalised states.
__global__ __launch_bounds__(kThreads) void merge_state_kernel(int rows, int D, const float* o_a,
                                                               const float* lse_a, const float* o_b,
                                                               const float* lse_b, float* o_out,
                                                               float* lse_out) {
  const int row = blockIdx.x;
  if (row >= rows) return;
  const float la = lse_a[row], lb = lse_b[row];
  const float m = fmaxf(la, lb);
  float wa = 0.f, wb = 0.f, lse = -INFINITY;
  if (m != -INFINITY) {
    wa = expf(la - m);
    wb = expf(lb - m);
    const float s = wa + wb;
    wa /= s;
    wb /= s;
    lse = m + logf(s);
  }
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    const size_t i = (size_t)row * D + d;
    o_out[i] = wa * o_a[i] + wb * o_b[i];
  }
  __syncthreads();
  if (threadIdx.x == 0) lse_out[row] = lse;
}

Params make_params(const d2sd_attn_args& a, const AttnPlan& plan, void* ws) {
  Params p{};
  p.q = a.q; p.k_cache = a.k_cache; p.v_cache = a.v_cache; p.page_table = a.page_table;
  p.ctx_len = a.ctx_len; p.k_tree = a.k_tree; p.v_tree = a.v_tree; p.node_indptr = a.node_indptr;
  p.anc_mask = a.anc_mask; p.out = a.out; p.lse = a.lse;
  const size_t rows = (size_t)a.total_nodes * a.num_qo_heads;
  // [normalised O in the input dtype][m][l] (fp32), each split-major
  char* w = static_cast<char*>(ws);
  const size_t o_bytes = (size_t)plan.n_ch_max * rows * kD * (a.dtype == D2SD_BF16 ? 2 : 4);
  p.ws_o = w;
  p.ws_m = w ? reinterpret_cast<float*>(w + o_bytes) : nullptr;
  p.ws_l = w ? p.ws_m + (size_t)plan.n_ch_max * rows : nullptr;
  p.batch = a.batch; p.hq = a.num_qo_heads; p.hkv = a.num_kv_heads; p.G = plan.G; p.stage = a.stage;
  p.total_nodes = a.total_nodes; p.max_nodes = a.max_nodes; p.max_ctx = a.max_ctx_len;
  p.num_pages = a.num_pages; p.max_pages = a.max_pages; p.mask_words = a.mask_words;
  p.split = plan.split; p.n_ch_max = plan.n_ch_max; p.n_rg_max = plan.n_rg_max;
  p.items = (int)plan.items;
  p.c2 = plan.scale * kLog2e;
  return p;
}

}  // namespace

hipError_t launch_cascade_attention(const d2sd_attn_args& a, const AttnPlan& plan, void* ws,
                                    hipStream_t stream, hipEvent_t (&ev)[3]) {
  const Params p = make_params(a, plan, ws);
  const int grid = (int)(((plan.items + 7) / 8) * 8);
  if (ev[0]) (void)hipEventRecord(ev[0], stream);
  if (a.dtype == D2SD_BF16 && plan.packed) {
    const long long wgs = (plan.tiles + pk::WAVES - 1) / pk::WAVES;
    const int pgrid = (int)(((wgs + 7) / 8) * 8);
    hipLaunchKernelGGL(cascade_bf16_packed_kernel, dim3(pgrid), dim3(pk::THREADS), 0, stream, p);
  } else if (a.dtype == D2SD_BF16 && plan.waves == kBf16WideWaves)
    hipLaunchKernelGGL(cascade_bf16_wide_kernel, dim3(grid), dim3(bf::Shape<kBf16WideWaves>::THREADS), 0, stream, p);
  else if (a.dtype == D2SD_BF16)
    hipLaunchKernelGGL(cascade_bf16_kernel, dim3(grid), dim3(bf::Shape<kBf16Waves>::THREADS), 0, stream, p);
  else
    hipLaunchKernelGGL(cascade_attention_kernel<float>, dim3(grid), dim3(kThreads), 0, stream, p);
  if (ev[1]) (void)hipEventRecord(ev[1], stream);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess && plan.n_ch_max > 1) {
    const int groups = merge_groups(plan.n_ch_max);
    const long long chunks = merge_chunks_per_request(a.max_nodes, a.num_qo_heads, groups);
    const dim3 mgrid((unsigned)(a.batch * chunks));
    if (a.dtype == D2SD_BF16) {
      if (groups > 1)
        hipLaunchKernelGGL((split_merge_kernel<__bf16, 4>), mgrid, dim3(kThreads), 0, stream, p, (int)chunks);
      else
        hipLaunchKernelGGL((split_merge_kernel<__bf16, 1>), mgrid, dim3(kThreads), 0, stream, p, (int)chunks);
    } else {
      if (groups > 1)
        hipLaunchKernelGGL((split_merge_kernel<float, 4>), mgrid, dim3(kThreads), 0, stream, p, (int)chunks);
      else
        hipLaunchKernelGGL((split_merge_kernel<float, 1>), mgrid, dim3(kThreads), 0, stream, p, (int)chunks);
    }
    e = hipGetLastError();
    if (ev[2]) (void)hipEventRecord(ev[2], stream);
  }
  return e;
}

hipError_t launch_noncascade_attention(const d2sd_attn_args& a, float scale, hipStream_t stream,
                                       hipEvent_t (&ev)[3]) {
  AttnPlan plan{};
  plan.G = a.num_qo_heads / a.num_kv_heads;
  plan.waves = kBf16Waves;
  plan.packed = false;
  plan.tiles = 0;
  plan.split = 1 << 30;  // whole context in one pass
  plan.n_ch_max = 1;
  plan.n_rg_max = 1;
  plan.items = (long long)a.batch * a.num_kv_heads * a.max_nodes;
  plan.scale = scale;
  const Params p = make_params(a, plan, nullptr);
  const int grid = (int)(((plan.items + 7) / 8) * 8);
  if (ev[0]) (void)hipEventRecord(ev[0], stream);
  if (a.dtype == D2SD_BF16)
    hipLaunchKernelGGL(noncascade_bf16_kernel, dim3(grid), dim3(bf::Shape<kBf16Waves>::THREADS), 0, stream, p);
  else
    hipLaunchKernelGGL(noncascade_attention_kernel<float>, dim3(grid), dim3(kThreads), 0, stream, p);
  if (ev[1]) (void)hipEventRecord(ev[1], stream);
  return hipGetLastError();
}

// ---- static scratch of the allocation-free entry point -------------------
// The split partial states of d2sd_cascade_verify_attention_noalloc live in
// this file-scope device array instead of a caller workspace. Each GPU the
// library runs on holds its own copy until the process ends. In host code
// `scratch` names a host-side stand-in, never the device memory: kernels get
// the address that hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) char scratch[kScratchBytes];

hipError_t scratch_address(void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));   // with `dev` current: its own copy
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

hipError_t launch_merge_state(int rows, int head_dim, const float* o_a, const float* lse_a,
                              const float* o_b, const float* lse_b, float* o_out, float* lse_out,
                              hipStream_t stream) {
  const int threads = head_dim >= 256 ? 256 : ((head_dim + 63) / 64) * 64;
  hipLaunchKernelGGL(merge_state_kernel, dim3(rows), dim3(threads), 0, stream, rows, head_dim, o_a,
                     lse_a, o_b, lse_b, o_out, lse_out);
  return hipGetLastError();
}

}  // namespace d2sd
