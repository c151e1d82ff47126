// Compaction of the accepted path's K/V rows into the paged cache, and the
// debug-time contract check, for gfx950.
//
// Keeping exactly the accepted tokens' keys/values is what turns a verified
// path into committed context (§1: the KV cache holds every committed token;
// rejected branches are dropped). One workgroup per (path position j,
// sequence b) copies node accept_idx[b][j]'s K and V rows (Hkv * D bf16 each)
// to cache position kv_len[b] + j with 16-byte vector moves.
#include "tv_internal.h"

namespace tv {
namespace {

constexpr int kCompactThreads = 128;

__global__ __launch_bounds__(kCompactThreads) void kv_compact_kernel(
    const uint16_t *__restrict__ k_tree, const uint16_t *__restrict__ v_tree,
    uint16_t *__restrict__ k_cache, uint16_t *__restrict__ v_cache,
    const int32_t *__restrict__ page_table, const int32_t *__restrict__ kv_len,
    const int32_t *__restrict__ accept_idx, const int32_t *__restrict__ accept_len, int N,
    int row_elems, int P, int p_shift, int max_pages, int num_pages) {
    const int j = blockIdx.x;
    const int b = blockIdx.y;
    if (j >= accept_len[b]) return;
    const int node = accept_idx[(size_t)b * N + j];
    const int pos = kv_len[b] + j;
    if (node < 0 || node >= N || pos < 0) return;
    const int slot_page = pos >> p_shift;
    if (slot_page >= max_pages) return;
    const int pg = page_table[(size_t)b * max_pages + slot_page];
    if (pg < 0 || pg >= num_pages) return;
    const size_t dst = (((size_t)pg << p_shift) + (pos & (P - 1))) * row_elems;
    const size_t src = ((size_t)b * N + node) * row_elems;
    const u16x8 *ks = reinterpret_cast<const u16x8 *>(k_tree + src);
    const u16x8 *vs = reinterpret_cast<const u16x8 *>(v_tree + src);
    u16x8 *kd = reinterpret_cast<u16x8 *>(k_cache + dst);
    u16x8 *vd = reinterpret_cast<u16x8 *>(v_cache + dst);
    for (int c = threadIdx.x; c < row_elems / 8; c += kCompactThreads) {
        kd[c] = ks[c];
        vd[c] = vs[c];
    }
}

__global__ __launch_bounds__(256) void validate_kernel(
    const int32_t *__restrict__ page_table, const int32_t *__restrict__ kv_len,
    const int32_t *__restrict__ parent, const int32_t *__restrict__ num_nodes, int B, int N,
    int P, int max_pages, int num_pages, int32_t *__restrict__ status_word) {
    __shared__ int flags;
    if (threadIdx.x == 0) flags = 0;
    __syncthreads();
    int f = 0;
    for (long idx = threadIdx.x; idx < (long)B * N; idx += blockDim.x) {
        const int b = (int)(idx / N), i = (int)(idx % N);
        if (num_nodes) {
            const int nb = num_nodes[b];
            if (nb < 0 || nb > N) { f |= 16; continue; }
            if (i >= nb) continue;                          // padding node: never read
        }
        const int pi = parent[idx];
        if (pi < -1 || pi >= i) f |= 1;
    }
    for (int b = threadIdx.x; b < B; b += blockDim.x) {
        const int L = kv_len[b];
        if (L < 0) { f |= 2; continue; }
        int nb = N;
        if (num_nodes) {
            nb = num_nodes[b];
            if (nb <= 0 || nb > N) continue;                // no pages are touched (or bit 4)
        }
        const long need = ((long)L + nb + P - 1) / P;     // prefix plus up to nb compacted rows
        if (need > max_pages) f |= 4;
        const long upto = need < max_pages ? need : max_pages;
        for (long k = 0; k < upto; ++k) {
            const int pg = page_table[(size_t)b * max_pages + k];
            if (pg < 0 || pg >= num_pages) f |= 8;
        }
    }
    if (f) atomicOr(&flags, f);
    __syncthreads();
    if (threadIdx.x == 0) *status_word = flags;
}

}  // namespace

hipError_t launch_kv_compact(const uint16_t *k_tree, const uint16_t *v_tree, uint16_t *k_cache,
                             uint16_t *v_cache, const int32_t *page_table, const int32_t *kv_len,
                             const int32_t *accept_idx, const int32_t *accept_len, int B, int N,
                             int Hkv, int D, int P, int max_pages, int num_pages, hipStream_t s) {
    if (B == 0) return hipSuccess;
    const int p_shift = __builtin_ctz((unsigned)P);
    return launch_kernel(kv_compact_kernel, dim3(N, B), dim3(kCompactThreads), s, k_tree, v_tree,
                         k_cache, v_cache, page_table, kv_len, accept_idx, accept_len, N, Hkv * D,
                         P, p_shift, max_pages, num_pages);
}

hipError_t launch_validate(const int32_t *page_table, const int32_t *kv_len,
                           const int32_t *parent, const int32_t *num_nodes, int B, int N, int P,
                           int max_pages, int num_pages, int32_t *status_word, hipStream_t s) {
    return launch_kernel(validate_kernel, dim3(1), dim3(256), s, page_table, kv_len, parent,
                         num_nodes, B, N, P, max_pages, num_pages, status_word);
}

}  // namespace tv
