// Internal declarations shared by the HIP sources of libtreeverify (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <tuple>
#include <type_traits>
#include <utility>

namespace tv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kNumXcd = 8;           // MI355X: 8 XCDs, workgroups dispatched round-robin
constexpr int kKeyTile = 64;         // keys per attention tile (two 32-key MFMA blocks)
constexpr int kRowsPerWave = 32;     // query rows per wave (MFMA N dimension)
constexpr int kMaxNodes = 256;
constexpr int kMaxBatchAttn = 1024;
constexpr int kTbMaxK = 16;          // tree builder: largest branch number
constexpr int kTbMaxSteps = 16;      // tree builder: most speculative steps

// Order-preserving key of a float: larger value -> larger key; NaN largest;
// -0 and +0 equal.
__device__ __forceinline__ unsigned int order_key(float x) {
    unsigned int u = __float_as_uint(x);
    if (x != x) return 0xFFFFFFFFu;
    if (x == 0.f) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// (value key, index) packed so that a plain unsigned maximum picks the larger
// value and, among equal values, the lower index.
__device__ __forceinline__ unsigned long long pack_key(unsigned int key, unsigned int idx) {
    return ((unsigned long long)key << 32) | (unsigned long long)(0xFFFFFFFFu - idx);
}

// Launch geometry and workspace layout of the tree builder.
struct TreeBuildPlan {
    int segs, seg_len;         // vocabulary segments per (sequence, step) row
    int chunks, chunk_len;     // hot-column chunks per frontier node (0 without hot tokens)
    int max_nodes;             // nodes of the unpruned tree: 1 + k + (S - 1) k^2
    size_t rows_bytes, parts_bytes, hot_logits_bytes, nodes_bytes, frontier_bytes;
};
TreeBuildPlan tree_build_plan(int B, int S, int V, int H, int k);

// Launch parameters of the tree-attention kernels (all sizes in elements).
struct AttnParams {
    const uint16_t *q, *k_tree, *v_tree, *k_cache, *v_cache;
    const int32_t *page_table, *kv_len, *parent;
    const int32_t *num_nodes;   // [B] node count per sequence, or null (N each)
    uint16_t *out;
    float *lse;
    uint16_t *ws_o;    // [num_wg * 2][rows_per_block][D] bf16 partial outputs (normalised)
    float *ws_ml;      // [num_wg * 2][rows_per_block][2] partial (max, sum)
    int32_t *ws_desc;  // [num_wg][4] per workgroup: the split unit it finishes (b, g, rb, first slot), b < 0 if none
    int B, N, Hq, Hkv, G, P, p_shift, max_pages, num_pages;
    int rows_per_block;          // query rows of one unit (the workgroup's waves x 32)
    int small_pages;             // pages shorter than one 1 KB load block of keys
    int narrow;                  // units of at most 16 rows: tiles shared out over the waves
    int setup_tiles;             // cost of starting a unit piece, in tiles (work balance)
    int num_wg;
    float scale_log2;            // softmax scale * log2(e)
    float scale;                 // softmax scale
};

// Workgroup -> logical index remap: the hardware hands consecutive workgroup
// ids to consecutive XCDs; give every XCD one contiguous run of logical ids
// so neighbouring work (which shares K/V rows) shares that XCD's L2.
__device__ __forceinline__ int xcd_contiguous_id(int hw_id, int n) {
    const int xcd = hw_id % kNumXcd;
    const int local = hw_id / kNumXcd;
    const int base = xcd * (n / kNumXcd) + min(xcd, n % kNumXcd);
    return base + local;
}

// Launch a kernel and return the runtime's status for this launch alone
// (hipGetLastError after hipLaunchKernelGGL would also report an error left
// behind by an unrelated earlier call of the caller's).
template <typename... KArgs, typename... Args>
inline hipError_t launch_kernel(void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t s,
                                Args &&...args) {
    static_assert(sizeof...(KArgs) == sizeof...(Args), "kernel argument count");
    std::tuple<std::decay_t<KArgs>...> held(std::forward<Args>(args)...);
    return std::apply(
        [&](auto &...a) {
            void *ptrs[] = {static_cast<void *>(&a)...};
            return hipLaunchKernel(reinterpret_cast<const void *>(kernel), grid, block, ptrs, 0, s);
        },
        held);
}

// Host-side launchers (defined next to their kernels).
hipError_t launch_tree_build(const float *logits, const int32_t *root_token,
                             const uint16_t *table, const int32_t *hot_vocab,
                             const int32_t *hot_index, const int32_t *accept_len, int r, int B,
                             int S, int V, int H, int k, int budget, int32_t *parent,
                             int32_t *token, float *joint, int32_t *num_nodes, void *workspace,
                             hipStream_t s);
hipError_t launch_tree_attention(const AttnParams &p, int head_dim, int waves, hipStream_t s);
hipError_t launch_argmax_accept(const float *logits, const int32_t *draft, const int32_t *parent,
                                const int32_t *num_nodes, int B, int N, int V, int segs,
                                int seg_len, int32_t *argmax_out,
                                int32_t *accept_len, int32_t *accept_idx, int32_t *bonus,
                                unsigned long long *ws, hipStream_t s);
// Greedy acceptance over per-node argmax keys: keys[(b * N + i) * segs + s].
hipError_t launch_accept(const unsigned long long *keys, int segs, const int32_t *draft,
                         const int32_t *parent, const int32_t *num_nodes, int B, int N,
                         int32_t *argmax_out, int32_t *accept_len, int32_t *accept_idx,
                         int32_t *bonus, hipStream_t s);
int lm_head_vocab_tiles(int V);
hipError_t launch_lm_head_argmax_accept(const uint16_t *hidden, const uint16_t *w,
                                        const int32_t *draft, const int32_t *parent,
                                        const int32_t *num_nodes, int B, int N, int V, int d,
                                        int32_t *argmax_out, int32_t *accept_len,
                                        int32_t *accept_idx, int32_t *bonus,
                                        unsigned long long *keys, hipStream_t s);
hipError_t launch_kv_compact(const uint16_t *k_tree, const uint16_t *v_tree, uint16_t *k_cache,
                             uint16_t *v_cache, const int32_t *page_table, const int32_t *kv_len,
                             const int32_t *accept_idx, const int32_t *accept_len, int B, int N,
                             int Hkv, int D, int P, int max_pages, int num_pages, hipStream_t s);
hipError_t launch_validate(const int32_t *page_table, const int32_t *kv_len,
                           const int32_t *parent, const int32_t *num_nodes, int B, int N, int P,
                           int max_pages, int num_pages, int32_t *status_word, hipStream_t s);

}  // namespace tv
