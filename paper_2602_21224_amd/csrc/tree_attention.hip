// Tree-masked attention over a paged KV prefix for gfx950 (MI355X).
//
// What is computed (the paper's tree-shaped verification attention, §2.1, with
// the tree mask of SpecInfer cited in §8, over the paged cache of §7.1): for
// every sequence b, KV head g and query row (node i, query head h of g's
// group), the softmax-weighted sum of values over the whole committed prefix
// plus node i's own root path.
//
// Work decomposition
//   * A "row block" is up to 256 query rows of one (b, g): row r is node r / G,
//     head g * G + r % G, so the G heads sharing a KV head are batched and every
//     K/V tile is read once for all of them (GQA grouping).
//   * A "unit" is one (b, g, row block). Its work is a list of 64-key tiles: the
//     prefix tiles, then the tree tiles (tree nodes 0 .. the block's last node).
//     All units' tiles are laid end to end and the workgroups take equal
//     contiguous shares, so ragged prefixes stay balanced. A workgroup that
//     covers a whole unit writes the output directly; a split unit leaves
//     per-piece (max, sum, numerator) partials that a second kernel merges with
//     the usual log-sum-exp rescaling.
//   * K and V tiles stream from HBM straight into a 4-stage LDS ring with
//     global_load_lds_dwordx4 (no register staging), three tiles ahead of the
//     one being computed. Each 256-byte row is stored with its 16-byte chunks
//     XOR-swizzled by the key index, so the MFMA operand reads below are free
//     of bank conflicts. Keys past the prefix, and tree slots past N, load a
//     harmless finite row (tree node 0) and are masked; the NaN-filled tail
//     slots of a cache page are never read.
//   * Each wave owns 32 query rows. Per 32-key half tile it computes
//     S^T = K * Q^T with v_mfma_f32_32x32x16_bf16 (keys on M, rows on N: a lane
//     holds 16 scores of one row, so a row max/sum needs one cross-half
//     exchange), masks, runs the online softmax in fp32 (base-2 exponent with
//     the scale folded into one FMA), and accumulates O^T = V^T * P^T with the
//     same instruction. V^T operands come from the row-major tile through
//     ds_read_b64_tr_b16, which transposes 4x16 blocks on the way out of LDS.
//   * Reads of the ring are inline assembly with explicit lgkmcnt waits tied to
//     the fragments they produce, and ring hand-off is s_waitcnt vmcnt(n) +
//     s_barrier, so the compiler never inserts a blanket wait for the
//     in-flight tile loads.
//   * Tree visibility is a per-node ancestor bit set (256 bits) built in LDS by
//     pointer doubling over the parent links; a masked score is replaced by -inf
//     (selected, never added).
#include "tv_internal.h"

namespace tv {
namespace {

#define LDS_AS __attribute__((address_space(3)))
#define GLOBAL_AS __attribute__((address_space(1)))

constexpr int KT = kKeyTile;           // 64 keys per tile
constexpr int NS = 4;                  // ring stages
constexpr int kPageCache = 1024;       // page ids cached in LDS per segment window
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLn2 = 0.693147180559945309f;
constexpr float kRescaleSlack = 8.f;   // keep a stale running max while new scores stay within 2^8 of it

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

template <int D>
struct Geo {
    static constexpr int kRowBytes = D * 2;
    static constexpr int kChunks = D / 8;                  // 16-byte chunks per row
    static constexpr int kTileBytes = KT * kRowBytes;      // one of K or V
    static constexpr int kStageBytes = 2 * kTileBytes;
    static constexpr int kBlocksPerTile = kTileBytes / 1024;
    static constexpr int kKeysPerBlock = 1024 / kRowBytes;
};

// Chunk swizzle of a key row: 16-byte chunk c of key k lives at position
// c ^ swz(k % chunks). swz swaps the two low bit-fields of the key so that both
// MFMA operand read patterns are free of LDS bank conflicts: 16 consecutive
// keys at one chunk (K fragments), and 4 consecutive keys x 4 adjacent chunks
// (the transposing V reads). It is a bit permutation, so swz(a ^ b) =
// swz(a) ^ swz(b).
template <int C>
__device__ __forceinline__ constexpr int swz(int k) {
    static_assert(C == 8 || C == 16, "rows of 64 or 128 bf16");
    return C == 16 ? (((k & 3) << 2) | ((k >> 2) & 3)) : (((k & 3) << 1) | ((k >> 2) & 1));
}

// Combine a per-row value held by lanes l and l ^ 32 (the two halves of a
// 32x32 MFMA tile column) without going through LDS.
__device__ __forceinline__ float halves_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// LDS objects are separate so the compiler can see that only `g_ring` is a
// target of the asynchronous tile loads.
__shared__ __attribute__((aligned(1024))) unsigned char g_ring[NS * Geo<128>::kStageBytes];
__shared__ unsigned long long g_anc[kMaxNodes][4];
__shared__ unsigned long long g_anc_alt[kMaxNodes][4];
__shared__ int g_par[kMaxNodes];
__shared__ int g_jump[2][kMaxNodes];
__shared__ int g_pages[kPageCache];
__shared__ int g_cum[kMaxBatchAttn + 1];

__device__ __forceinline__ unsigned lds_addr(const void *p) {
    return (unsigned)(size_t)(const LDS_AS void *)p;
}

__device__ __forceinline__ int clamp_len(int L, const AttnParams &p) {
    const int cap = p.max_pages << p.p_shift;
    return L < 0 ? 0 : (L > cap ? cap : L);
}

__device__ __forceinline__ int tree_tiles_of_block(int rb, const AttnParams &p) {
    const int last_row = min((rb + 1) * p.rows_per_block, p.rows) - 1;
    const int jmax = last_row / p.G + 1;                  // nodes 0 .. jmax-1 may be ancestors
    return (jmax + KT - 1) / KT;
}

__device__ __forceinline__ int tiles_of_sequence(int b, const AttnParams &p) {
    const int L = clamp_len(p.kv_len[b], p);
    return p.Hkv * (p.row_blocks * ((L + KT - 1) / KT) + p.tree_tiles_all_blocks);
}

// Explicit LDS wait for reads issued through inline assembly; `tie` makes a
// fragment's later uses depend on the wait (volatile asm keeps its order).
template <int N>
__device__ __forceinline__ void lds_wait() {
    asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}
template <typename T>
__device__ __forceinline__ void tie(T &x) {
    asm volatile("" : "+v"(x));
}

__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// s_waitcnt through the builtin, so the compiler's own wait insertion knows
// about it. gfx9 encoding: vmcnt in [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8].
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt is a 6-bit field");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ void wait_tile_loads(int newer_tiles, int loads_per_tile) {
    // At most newer_tiles * loads_per_tile later loads may stay in flight; a
    // count without its own case waits for the next smaller one (stricter).
    const int n = newer_tiles * loads_per_tile;
    if (n >= 32) wait_vmcnt<32>();
    else if (n >= 16) wait_vmcnt<16>();
    else if (n >= 8) wait_vmcnt<8>();
    else if (n >= 4) wait_vmcnt<4>();
    else if (n >= 2) wait_vmcnt<2>();
    else wait_vmcnt<0>();
}

// Exclusive prefix sum of per-sequence tile counts into g_cum[0..B].
template <int NT>
__device__ void build_cumulative(const AttnParams &p) {
    const int tid = threadIdx.x;
    const int per = (p.B + NT - 1) / NT;
    const int b0 = tid * per;
    const int b1 = min(b0 + per, p.B);
    int local = 0;
    for (int b = b0; b < b1; ++b) local += tiles_of_sequence(b, p);
    int *scan = &g_jump[0][0];            // 2 * kMaxNodes >= NT ints of scratch
    scan[tid] = local;
    __syncthreads();
    for (int off = 1; off < NT; off <<= 1) {
        const int v = tid >= off ? scan[tid - off] : 0;
        __syncthreads();
        scan[tid] += v;
        __syncthreads();
    }
    int run = scan[tid] - local;
    for (int b = b0; b < b1; ++b) {
        g_cum[b] = run;
        run += tiles_of_sequence(b, p);
    }
    if (tid == NT - 1) g_cum[p.B] = scan[NT - 1];
    __syncthreads();
}

// Segment set-up, part 1: page ids of pages [first, first + kPageCache) of
// sequence b (as far as it has them) into g_pages, and the parent links of
// sequence b into g_par. All loads are issued before any is waited for.
template <int NT>
__device__ void load_pages_and_parents(const AttnParams &p, int b, int first, int npages,
                                       bool want_pages, bool want_parents) {
    constexpr int PPT = (kPageCache + NT - 1) / NT;
    const int tid = threadIdx.x;
    const int n = want_pages ? min(kPageCache, npages - first) : 0;
    int pg[PPT];
    #pragma unroll
    for (int k = 0; k < PPT; ++k) {
        const int i = tid + k * NT;
        pg[k] = i < n ? p.page_table[(size_t)b * p.max_pages + first + i] : -1;
    }
    int par[(kMaxNodes + NT - 1) / NT];
    #pragma unroll
    for (int k = 0; k < (kMaxNodes + NT - 1) / NT; ++k) {
        const int i = tid + k * NT;
        par[k] = (want_parents && i < p.N) ? p.parent[(size_t)b * p.N + i] : -1;
    }
    #pragma unroll
    for (int k = 0; k < PPT; ++k) {
        const int i = tid + k * NT;
        if (i < n) g_pages[i] = (pg[k] >= 0 && pg[k] < p.num_pages) ? pg[k] : -1;
    }
    #pragma unroll
    for (int k = 0; k < (kMaxNodes + NT - 1) / NT; ++k) {
        const int i = tid + k * NT;
        if (want_parents && i < p.N) {
            const int pi = par[k];
            g_par[i] = (pi < -1 || pi >= i) ? -1 : pi;   // contract violation: treat as a root
        }
    }
    __syncthreads();
}

// Segment set-up, part 2: ancestor bit sets of the N nodes (from g_par) by
// pointer doubling: after round k a node's set holds every ancestor within
// distance < 2^k. Runs while the first tiles are in flight. Result in g_anc.
template <int NT>
__device__ void build_ancestor_masks(const AttnParams &p) {
    const int tid = threadIdx.x;
    for (int i = tid; i < p.N; i += NT) {
        #pragma unroll
        for (int w = 0; w < 4; ++w) g_anc[i][w] = (w == (i >> 6)) ? (1ull << (i & 63)) : 0ull;
        g_jump[0][i] = g_par[i];
    }
    __syncthreads();
    int cur = 0;
    for (int round = 0; round < 8; ++round) {
        unsigned long long(*src)[4] = cur == 0 ? g_anc : g_anc_alt;
        unsigned long long(*dst)[4] = cur == 0 ? g_anc_alt : g_anc;
        int more = 0;
        for (int i = tid; i < p.N; i += NT) {
            const int j = g_jump[cur][i];
            if (j >= 0) {
                #pragma unroll
                for (int w = 0; w < 4; ++w) dst[i][w] = src[i][w] | src[j][w];
                const int jj = g_jump[cur][j];
                g_jump[cur ^ 1][i] = jj;
                more |= jj >= 0;
            } else {
                #pragma unroll
                for (int w = 0; w < 4; ++w) dst[i][w] = src[i][w];
                g_jump[cur ^ 1][i] = -1;
            }
        }
        cur ^= 1;
        if (!__syncthreads_or(more)) break;
    }
    if (cur == 1) {
        for (int i = tid; i < p.N; i += NT)
            #pragma unroll
            for (int w = 0; w < 4; ++w) g_anc[i][w] = g_anc_alt[i][w];
        __syncthreads();
    }
}

template <int D, int NW>
struct TileIssue {
    using Gm = Geo<D>;
    static constexpr int kLoadsPerWave = 2 * Gm::kBlocksPerTile / NW;
    static constexpr int KPB = Gm::kKeysPerBlock;     // keys per 1 KB load block
    static constexpr int C = Gm::kChunks;

    int kib;                                          // this lane's key within a block
    unsigned row_off;                                 // kib * key row stride (bytes)
    unsigned chunk_off[kLoadsPerWave];                // swizzled chunk offset per load

    __device__ __forceinline__ void init(int wave_u, int lane, unsigned row_stride) {
        kib = lane / C;
        row_off = kib * row_stride;
        #pragma unroll
        for (int i = 0; i < kLoadsPerWave; ++i) {
            const int kb = (wave_u * kLoadsPerWave + i) % Gm::kBlocksPerTile;
            chunk_off[i] = (unsigned)(((lane % C) ^ swz<C>((kb * KPB + kib) % C)) * 16);
        }
    }

    // Issue the direct-to-LDS loads of tile t of unit (b, g) into ring stage
    // `stage`. A load block covers KPB consecutive keys; when a page holds at
    // least KPB keys they share one page, so the block's base address is
    // wave-uniform (scalar math) and lanes only add their row/chunk offset.
    // Rows that do not exist (past the prefix, past N) re-read the block's
    // first row, or tree node 0 when the whole block is past the end.
    __device__ __forceinline__ void issue(const AttnParams &p, int b, int g, int L, int ntp,
                                          int t, int stage, int page_first, int wave_u) const {
        const uint16_t *safe_k = p.k_tree + ((size_t)b * p.N * p.Hkv + g) * D;
        const uint16_t *safe_v = p.v_tree + ((size_t)b * p.N * p.Hkv + g) * D;
        #pragma unroll
        for (int i = 0; i < kLoadsPerWave; ++i) {
            const int blk = wave_u * kLoadsPerWave + i;                 // wave-uniform
            const bool is_v = blk >= Gm::kBlocksPerTile;
            const int kb = is_v ? blk - Gm::kBlocksPerTile : blk;
            const uint16_t *base = is_v ? safe_v : safe_k;
            const char *addr;
            if (t < ntp) {
                const int pos0 = t * KT + kb * KPB;
                const int n_valid = min(max(L - pos0, 0), KPB);
                if (!p.small_pages) {
                    int pg = -1;
                    if (n_valid > 0)
                        pg = __builtin_amdgcn_readfirstlane(g_pages[(pos0 >> p.p_shift) - page_first]);
                    const bool ok = pg >= 0;
                    if (ok)
                        base = (is_v ? p.v_cache : p.k_cache) +
                               ((((size_t)pg << p.p_shift) + (pos0 & (p.P - 1))) * p.Hkv + g) * D;
                    addr = reinterpret_cast<const char *>(base) +
                           ((ok && kib < n_valid ? row_off : 0u) + chunk_off[i]);
                } else {
                    // pages shorter than a load block: every lane finds its own page
                    const int pos = pos0 + kib;
                    const uint16_t *row = base;
                    if (kib < n_valid) {
                        const int pg = g_pages[(pos >> p.p_shift) - page_first];
                        if (pg >= 0)
                            row = (is_v ? p.v_cache : p.k_cache) +
                                  ((((size_t)pg << p.p_shift) + (pos & (p.P - 1))) * p.Hkv + g) * D;
                    }
                    addr = reinterpret_cast<const char *>(row) + chunk_off[i];
                }
            } else {
                const int j0 = (t - ntp) * KT + kb * KPB;
                const int n_valid = min(max(p.N - j0, 0), KPB);
                if (n_valid > 0) base += (size_t)j0 * p.Hkv * D;
                addr = reinterpret_cast<const char *>(base) + ((kib < n_valid ? row_off : 0u) + chunk_off[i]);
            }
            unsigned char *dst = g_ring + stage * Gm::kStageBytes + (is_v ? Gm::kTileBytes : 0) + kb * 1024;
            __builtin_amdgcn_global_load_lds((const GLOBAL_AS void *)addr, (LDS_AS void *)dst, 16, 0, 0);
        }
    }
};

template <int D, int NW>
__global__ __launch_bounds__(NW * kWave) void tree_attention_kernel(AttnParams p) {
    using Gm = Geo<D>;
    using Issue = TileIssue<D, NW>;
    constexpr int NT = NW * kWave;
    constexpr int NKS = D / 16;     // MFMA k-steps over the head dim
    constexpr int NDT = D / 32;     // 32-wide head-dim tiles of the output
    constexpr int LPW = Issue::kLoadsPerWave;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave_u = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int half = lane >> 5;
    const int col = lane & 31;
    const int w = xcd_contiguous_id(blockIdx.x, p.num_wg);

    build_cumulative<NT>(p);
    if (w == 0)
        for (int b = tid; b <= p.B; b += NT) p.ws_cum[b] = g_cum[b];

    const int total = g_cum[p.B];
    const int share = (total + p.num_wg - 1) / p.num_wg;
    const int start = min(w * share, total);
    const int end = min(start + share, total);
    const unsigned ring_base = lds_addr(g_ring);
    Issue ld;
    ld.init(wave_u, lane, (unsigned)(p.Hkv * D * 2));

    // lane-constant parts of the LDS fragment addresses (see swz)
    const unsigned k_lane = col * Gm::kRowBytes + ((half ^ swz<Gm::kChunks>(col % Gm::kChunks)) << 4);
    const int va = ((lane >> 4) & 1) * 2 + ((lane & 3) >> 1);
    const int vb = half * 4 + ((lane & 15) >> 2);
    const unsigned v_lane = vb * Gm::kRowBytes + ((va ^ swz<Gm::kChunks>(vb)) << 4) + (lane & 1) * 8;

    int pos = start;
    int seg_no = 0;
    while (pos < end) {
        // ---- locate the unit holding tile `pos`
        int lo = 0, hi = p.B - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (g_cum[mid] <= pos) lo = mid; else hi = mid - 1;
        }
        const int b = lo;
        const int L = clamp_len(p.kv_len[b], p);
        const int ntp = (L + KT - 1) / KT;
        const int per_g = p.row_blocks * ntp + p.tree_tiles_all_blocks;
        int off = pos - g_cum[b];
        const int g = off / per_g;
        off -= g * per_g;
        int rb = 0;
        int ulen = ntp + tree_tiles_of_block(0, p);
        while (off >= ulen) {
            off -= ulen;
            ++rb;
            ulen = ntp + tree_tiles_of_block(rb, p);
        }
        const int t_begin = off;
        const int t_end = min(ulen, off + (end - pos));
        const bool complete = (t_begin == 0 && t_end == ulen);

        // ---- this wave's 32 query rows: Q fragments stay in registers
        const int row = rb * p.rows_per_block + wave_u * kRowsPerWave + col;
        const bool row_ok = row < p.rows;
        const int node = row_ok ? row / p.G : 0;
        const int hq = g * p.G + (row_ok ? row % p.G : 0);
        bf16x8 qf[NKS];
        {
            const uint16_t *qp = p.q + (((size_t)b * p.N + node) * p.Hq + hq) * D + half * 8;
            #pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
                u16x8 v = row_ok ? *reinterpret_cast<const u16x8 *>(qp + ks * 16)
                                 : u16x8{0, 0, 0, 0, 0, 0, 0, 0};
                qf[ks] = __builtin_bit_cast(bf16x8, v);
            }
        }

        // ---- page ids and parent links (one round trip), then the first tiles
        const int npages = (L + p.P - 1) >> p.p_shift;
        int page_first = (t_begin * KT) >> p.p_shift;
        const bool has_tree = t_end > ntp;
        load_pages_and_parents<NT>(p, b, page_first, npages, t_begin < ntp, has_tree);

        f32x16 o[NDT];
        #pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
            #pragma unroll
            for (int r = 0; r < 16; ++r) o[dt][r] = 0.f;
        float m_run = kNegInf;          // running max in raw score units
        float l_run = 0.f;

        __builtin_amdgcn_s_waitcnt(0);  // Q, ids and earlier stores drained
        #pragma unroll
        for (int k = 0; k < NS - 1; ++k)
            if (t_begin + k < t_end)
                ld.issue(p, b, g, L, ntp, t_begin + k, (t_begin + k) % NS, page_first, wave_u);
        if (has_tree) build_ancestor_masks<NT>(p);   // overlaps the loads above

        for (int t = t_begin; t < t_end; ++t) {
            const int stage = t % NS;
            wait_tile_loads(min(NS - 2, t_end - 1 - t), LPW);
            lds_barrier();
            const int tn = t + NS - 1;
            if (tn < t_end) {
                if (tn < ntp) {
                    const int last_page = (min(tn * KT + KT, L) - 1) >> p.p_shift;
                    if (last_page >= page_first + kPageCache) {
                        page_first = (tn * KT) >> p.p_shift;
                        wait_vmcnt<0>();
                        load_pages_and_parents<NT>(p, b, page_first, npages, true, false);
                    }
                }
                ld.issue(p, b, g, L, ntp, tn, tn % NS, page_first, wave_u);
            }

            const unsigned kaddr = ring_base + stage * Gm::kStageBytes + k_lane;
            const unsigned vaddr = ring_base + stage * Gm::kStageBytes + Gm::kTileBytes + v_lane;

            // ---- scores of both 32-key halves: S^T[key][row] = K[key][:] . Q[row][:].
            // At most 15 LDS reads can be tracked in flight; each half's K reads
            // are issued while the previous MFMAs execute.
            f32x16 s[2];
            #pragma unroll
            for (int hf = 0; hf < 2; ++hf)
                #pragma unroll
                for (int r = 0; r < 16; ++r) s[hf][r] = 0.f;
            #pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                u32x4 kf[NKS];
                #pragma unroll
                for (int ks = 0; ks < NKS; ++ks)
                    asm volatile("ds_read_b128 %0, %1 offset:%2"
                                 : "=v"(kf[ks])
                                 : "v"(kaddr ^ ((unsigned)ks << 5)), "i"(hf * 32 * Gm::kRowBytes));
                constexpr int H = NKS / 2;
                lds_wait<H>();
                #pragma unroll
                for (int ks = 0; ks < H; ++ks) {
                    tie(kf[ks]);
                    s[hf] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, kf[ks]), qf[ks], s[hf], 0, 0, 0);
                }
                lds_wait<0>();
                #pragma unroll
                for (int ks = H; ks < NKS; ++ks) {
                    tie(kf[ks]);
                    s[hf] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, kf[ks]), qf[ks], s[hf], 0, 0, 0);
                }
            }
            // V fragments (transposing reads) of the first half; they arrive during
            // the mask and softmax below
            u32x2 vf[2][2][NDT][2];        // [half][kstep][dt][rr]
            auto read_v = [&](int hf, int kstep) {
                #pragma unroll
                for (int dt = 0; dt < NDT; ++dt)
                    #pragma unroll
                    for (int rr = 0; rr < 2; ++rr) {
                        const unsigned flip =
                            (unsigned)((dt * 4) ^ swz<Gm::kChunks>((rr * 8) % Gm::kChunks)) << 4;
                        const unsigned a = vaddr ^ flip;
                        if (hf == 0 && kstep == 0)
                            asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(vf[0][0][dt][rr])
                                         : "v"(a), "i"((rr * 8) * Gm::kRowBytes));
                        else if (hf == 0)
                            asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(vf[0][1][dt][rr])
                                         : "v"(a), "i"((16 + rr * 8) * Gm::kRowBytes));
                        else if (kstep == 0)
                            asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(vf[1][0][dt][rr])
                                         : "v"(a), "i"((32 + rr * 8) * Gm::kRowBytes));
                        else
                            asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(vf[1][1][dt][rr])
                                         : "v"(a), "i"((48 + rr * 8) * Gm::kRowBytes));
                    }
            };
            read_v(0, 0);
            read_v(0, 1);

            // ---- masks (only the tile that crosses the prefix end, and tree tiles).
            // Lane holds keys hf*32 + (r/4)*8 + half*4 + r%4 of row `col`.
            if (t < ntp) {
                const int lim = L - t * KT - half * 4;          // keys >= lim are past the prefix
                if (lim < 64) {
                    #pragma unroll
                    for (int hf = 0; hf < 2; ++hf)
                        #pragma unroll
                        for (int r = 0; r < 16; ++r)
                            if (hf * 32 + (r >> 2) * 8 + (r & 3) >= lim) s[hf][r] = kNegInf;
                }
            } else {
                const unsigned long long vis = g_anc[node][t - ntp] >> (half * 4);
                #pragma unroll
                for (int hf = 0; hf < 2; ++hf)
                    #pragma unroll
                    for (int r = 0; r < 16; ++r)
                        if (!((vis >> (hf * 32 + (r >> 2) * 8 + (r & 3))) & 1ull)) s[hf][r] = kNegInf;
            }

            // ---- online softmax over the whole tile. The running max is only
            // raised when a score exceeds it by more than kRescaleSlack (log2
            // units), so O is rarely rescaled.
            float tmax = fmaxf(s[0][0], s[1][0]);
            #pragma unroll
            for (int r = 1; r < 16; ++r) tmax = fmaxf(tmax, fmaxf(s[0][r], s[1][r]));
            tmax = halves_max(tmax);
            const bool raise = tmax * p.scale_log2 > m_run * p.scale_log2 + kRescaleSlack;
            if (__any(raise)) {
                const float m_new = raise ? tmax : m_run;
                const float alpha = (m_run == kNegInf) ? 0.f
                                    : __builtin_amdgcn_exp2f((m_run - m_new) * p.scale_log2);
                l_run *= alpha;
                #pragma unroll
                for (int dt = 0; dt < NDT; ++dt)
                    #pragma unroll
                    for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
                m_run = m_new;
            }
            const float msc = (m_run == kNegInf) ? 0.f : m_run * p.scale_log2;

            // P for the first half
            bf16x8 pb[2][2];
            float psum = 0.f;
            #pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(s[0][r], p.scale_log2, -msc));
                psum += e;
                pb[0][r >> 3][r & 7] = (__bf16)e;
            }
            lds_wait<0>();                    // the first half's V fragments are in
            #pragma unroll
            for (int kstep = 0; kstep < 2; ++kstep)
                #pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    tie(vf[0][kstep][dt][0]);
                    tie(vf[0][kstep][dt][1]);
                }
            read_v(1, 0);
            // PV of the first half interleaved with P of the second half
            #pragma unroll
            for (int kstep = 0; kstep < 2; ++kstep) {
                if (kstep == 1) read_v(1, 1);
                #pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    const u32x4 a = {vf[0][kstep][dt][0][0], vf[0][kstep][dt][0][1],
                                     vf[0][kstep][dt][1][0], vf[0][kstep][dt][1][1]};
                    o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, a), pb[0][kstep], o[dt], 0, 0, 0);
                }
            }
            #pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(s[1][r], p.scale_log2, -msc));
                psum += e;
                pb[1][r >> 3][r & 7] = (__bf16)e;
            }
            #pragma unroll
            for (int i = 0; i < NDT; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
                __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);   // then VALU work
            }
            l_run += psum;
            #pragma unroll
            for (int kstep = 0; kstep < 2; ++kstep) {
                if (kstep == 0) lds_wait<2 * NDT>(); else lds_wait<0>();
                #pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    tie(vf[1][kstep][dt][0]);
                    tie(vf[1][kstep][dt][1]);
                    const u32x4 a = {vf[1][kstep][dt][0][0], vf[1][kstep][dt][0][1],
                                     vf[1][kstep][dt][1][0], vf[1][kstep][dt][1][1]};
                    o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, a), pb[1][kstep], o[dt], 0, 0, 0);
                }
            }
        }

        // ---- finish the segment
        const float l_tot = halves_sum(l_run);
        if (complete) {
            if (row_ok) {
                const float inv = 1.f / l_tot;
                uint16_t *op = p.out + (((size_t)b * p.N + node) * p.Hq + hq) * D;
                #pragma unroll
                for (int dt = 0; dt < NDT; ++dt)
                    #pragma unroll
                    for (int q4 = 0; q4 < 4; ++q4) {
                        bf16x4 v;
                        #pragma unroll
                        for (int i = 0; i < 4; ++i) v[i] = (__bf16)(o[dt][q4 * 4 + i] * inv);
                        *reinterpret_cast<bf16x4 *>(op + dt * 32 + q4 * 8 + half * 4) = v;
                    }
                if (p.lse && half == 0)
                    p.lse[((size_t)b * p.N + node) * p.Hq + hq] =
                        m_run * p.scale + __builtin_amdgcn_logf(l_tot) * kLn2;
            }
        } else {
            const int slot = w * 2 + (seg_no == 0 ? 0 : 1);
            const int rloc = wave_u * kRowsPerWave + col;
            float *po = p.ws_o + ((size_t)slot * p.rows_per_block + rloc) * D;
            #pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
                #pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    f32x4 v = {o[dt][q4 * 4 + 0], o[dt][q4 * 4 + 1], o[dt][q4 * 4 + 2], o[dt][q4 * 4 + 3]};
                    *reinterpret_cast<f32x4 *>(po + dt * 32 + q4 * 8 + half * 4) = v;
                }
            if (half == 0) {
                float *pm = p.ws_ml + ((size_t)slot * p.rows_per_block + rloc) * 2;
                pm[0] = (m_run == kNegInf) ? kNegInf : m_run * p.scale_log2;
                pm[1] = l_tot;
            }
        }
        pos += t_end - t_begin;
        ++seg_no;
        __syncthreads();
    }
}

// Merge the partials of every unit that more than one workgroup worked on:
// one thread per (row, 4 head-dim lanes) of the unit.
template <int D>
__global__ __launch_bounds__(256) void tree_attention_merge_kernel(AttnParams p) {
    constexpr int D4 = D / 4;
    constexpr int kRowsPerWg = 256 / D4;
    const int chunks = (p.rows_per_block + kRowsPerWg - 1) / kRowsPerWg;
    const int unit = blockIdx.x / chunks;
    const int rchunk = blockIdx.x % chunks;
    const int rb = unit % p.row_blocks;
    const int g = (unit / p.row_blocks) % p.Hkv;
    const int b = unit / (p.row_blocks * p.Hkv);
    const int total = p.ws_cum[p.B];
    const int share = (total + p.num_wg - 1) / p.num_wg;
    const int L = clamp_len(p.kv_len[b], p);
    const int ntp = (L + KT - 1) / KT;
    int ustart = p.ws_cum[b] + g * (p.row_blocks * ntp + p.tree_tiles_all_blocks);
    for (int r = 0; r < rb; ++r) ustart += ntp + tree_tiles_of_block(r, p);
    const int ulen = ntp + tree_tiles_of_block(rb, p);
    const int wf = ustart / share;
    const int wl = (ustart + ulen - 1) / share;
    if (wf == wl) return;

    const int rl = rchunk * kRowsPerWg + threadIdx.x / D4;
    const int d4 = threadIdx.x % D4;
    const int row = rb * p.rows_per_block + rl;
    if (rl >= p.rows_per_block || row >= p.rows) return;

    float M = kNegInf;
    for (int w = wf; w <= wl; ++w) {
        const int slot = w * 2 + (ustart <= w * share ? 0 : 1);
        M = fmaxf(M, p.ws_ml[((size_t)slot * p.rows_per_block + rl) * 2]);
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    float den = 0.f;
    for (int w = wf; w <= wl; ++w) {
        const int slot = w * 2 + (ustart <= w * share ? 0 : 1);
        const float *pm = p.ws_ml + ((size_t)slot * p.rows_per_block + rl) * 2;
        const float wt = (pm[0] == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(pm[0] - M);
        den += wt * pm[1];
        const f32x4 v = *reinterpret_cast<const f32x4 *>(
            p.ws_o + ((size_t)slot * p.rows_per_block + rl) * D + d4 * 4);
        acc += wt * v;
    }
    const int node = row / p.G;
    const int hq = g * p.G + row % p.G;
    const float inv = den > 0.f ? 1.f / den : 0.f;
    bf16x4 v;
    #pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = (__bf16)(acc[i] * inv);
    *reinterpret_cast<bf16x4 *>(p.out + (((size_t)b * p.N + node) * p.Hq + hq) * D + d4 * 4) = v;
    if (p.lse && d4 == 0)
        p.lse[((size_t)b * p.N + node) * p.Hq + hq] = (M + __builtin_amdgcn_logf(den)) * kLn2;
}

template <int D, int NW>
hipError_t launch_dn(const AttnParams &p, hipStream_t s) {
    hipLaunchKernelGGL((tree_attention_kernel<D, NW>), dim3(p.num_wg), dim3(NW * kWave), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (p.num_wg > 1) {
        constexpr int kRowsPerWg = 256 / (D / 4);
        const int chunks = (p.rows_per_block + kRowsPerWg - 1) / kRowsPerWg;
        hipLaunchKernelGGL((tree_attention_merge_kernel<D>),
                           dim3(p.B * p.Hkv * p.row_blocks * chunks), dim3(256), 0, s, p);
        e = hipGetLastError();
    }
    return e;
}

template <int D>
hipError_t launch_d(const AttnParams &p, int waves, hipStream_t s) {
    switch (waves) {
        case 1: return launch_dn<D, 1>(p, s);
        case 2: return launch_dn<D, 2>(p, s);
        case 4: return launch_dn<D, 4>(p, s);
        case 8: return launch_dn<D, 8>(p, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_tree_attention(const AttnParams &p, int head_dim, int waves, hipStream_t s) {
    if (head_dim == 64) return launch_d<64>(p, waves, s);
    if (head_dim == 128) return launch_d<128>(p, waves, s);
    return hipErrorInvalidValue;
}

}  // namespace tv
