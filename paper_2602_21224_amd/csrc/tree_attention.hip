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
//     per-piece partials (max and sum in fp32, the piece's own normalised
//     output in bf16) that a second kernel merges with the usual log-sum-exp
//     rescaling.
//   * K and V tiles stream from HBM straight into a 4-stage LDS ring with
//     global_load_lds_dwordx4 (no register staging). Each 256-byte row is
//     stored with its 16-byte chunks XOR-swizzled by the key index, so the
//     MFMA operand reads below are free of bank conflicts. Keys past the
//     prefix, and tree slots past N, load a harmless finite row (tree node 0)
//     and are masked; the NaN-filled tail slots of a cache page are never read.
//   * Each wave owns 32 query rows; the workgroup's 8 waves step through the
//     tiles together, one workgroup barrier per 64-key tile ("period"). In
//     period j every wave computes S^T = K_j Q^T with
//     v_mfma_f32_32x32x16_bf16 (keys on M, rows on N: a lane holds 16 scores
//     of one row, so a row max/sum needs one cross-half exchange) and
//     O^T += V_{j-1}^T P_{j-1}^T with the same instruction, and puts the
//     softmax work (mask, max, fp32 exponentials in base 2 with the scale
//     folded into one FMA, bf16 P^T) between those MFMAs, so that one wave's
//     matrix and vector work overlap. V^T operands come from the row-major
//     tile through ds_read_b64_tr_b16, which transposes 4x16 blocks on the
//     way out of LDS.
//   * At the end of period j each wave issues its share of K_{j+3} and
//     V_{j+2} in one burst: DMA writes into LDS slow down every wave's operand
//     reads, and a single burst per period disturbs them least. Each load is
//     issued about three periods before it is read.
//   * Reads of the ring are inline assembly with explicit lgkmcnt waits tied to
//     the fragments they produce, and ring hand-off is s_waitcnt vmcnt(n) +
//     s_barrier, so the compiler never inserts a blanket wait for the
//     in-flight tile loads.
//   * Tree visibility is a per-node ancestor bit set (256 bits) in LDS, built
//     by one wave while the first tiles load: for trees of up to 64 nodes each
//     lane follows its node's parent links through cross-lane shuffles, larger
//     trees use pointer doubling in LDS. A masked score is replaced by -inf
//     (selected, never added).
#include "tv_internal.h"

namespace tv {
namespace {

#define LDS_AS __attribute__((address_space(3)))
#define GLOBAL_AS __attribute__((address_space(1)))
#define CONST_AS __attribute__((address_space(4)))

constexpr int KT = kKeyTile;           // 64 keys per tile
constexpr int NS = 4;                  // ring stages (a power of two: stage = tile & (NS - 1))
constexpr int kPageCache = 512;        // page ids cached in LDS per segment window
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
// Maximum of three values in one instruction (scores are never signalling NaNs).
__device__ __forceinline__ float max3(float a, float b, float c) {
    float r;
    asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}
__device__ __forceinline__ float halves_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// The same over lanes l, l ^ 16, l ^ 32 and l ^ 48 (the four 16-lane rows of a
// 16x16 MFMA tile's column), by the row-pair swap and then the half-wave swap.
__device__ __forceinline__ float rows_max(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return halves_max(fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1])));
}
__device__ __forceinline__ float rows_sum(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return halves_sum(__uint_as_float(r[0]) + __uint_as_float(r[1]));
}

// LDS objects are separate so the compiler can see that only `g_ring` is a
// target of the asynchronous tile loads.
__shared__ __attribute__((aligned(1024))) unsigned char g_ring[NS * Geo<128>::kStageBytes];
__shared__ unsigned long long g_anc[kMaxNodes][4];
__shared__ unsigned long long g_anc_alt[kMaxNodes][4];
__shared__ int g_jump[2][kMaxNodes];
__shared__ int g_pages[kPageCache];
__shared__ int g_cum[kMaxBatchAttn + 1];
__shared__ int g_len[kMaxBatchAttn];     // clamped prefix length per sequence
__shared__ unsigned short g_nn[kMaxBatchAttn];   // node count per sequence

__device__ __forceinline__ unsigned lds_addr(const void *p) {
    return (unsigned)(size_t)(const LDS_AS void *)p;
}

__device__ __forceinline__ int clamp_len(int L, const AttnParams &p) {
    const int cap = p.max_pages << p.p_shift;
    return L < 0 ? 0 : (L > cap ? cap : L);
}

// Tree tiles row block rb of a sequence with `rows` query rows must visit.
__device__ __forceinline__ int tree_tiles_of_block(int rb, int rows, const AttnParams &p) {
    const int last_row = min((rb + 1) * p.rows_per_block, rows) - 1;
    const int jmax = last_row / p.G + 1;                  // nodes 0 .. jmax-1 may be ancestors
    return (jmax + KT - 1) / KT;
}

__device__ __forceinline__ int row_blocks_of(int rows, const AttnParams &p) {
    return (rows + p.rows_per_block - 1) / p.rows_per_block;
}

// Virtual tiles of one KV head of a sequence with ntp prefix tiles and `rows`
// query rows: per row block the set-up tiles, the prefix and its tree tiles.
__device__ __forceinline__ int tiles_per_head(int ntp, int rows, const AttnParams &p) {
    int t = 0;
    for (int rb = 0; rb < row_blocks_of(rows, p); ++rb)
        t += p.setup_tiles + ntp + tree_tiles_of_block(rb, rows, p);
    return t;
}

__device__ __forceinline__ int nodes_of(int b, const AttnParams &p) {
    if (!p.num_nodes) return p.N;
    const int n = p.num_nodes[b];
    return n < 0 ? 0 : (n > p.N ? p.N : n);
}

// Work of sequence b in "virtual" tiles: every unit counts setup_tiles in
// front of its real tiles (the cost of starting a piece: its set-up and its
// pipeline fill), so that equal shares of virtual tiles balance the work of
// workgroups that start new units against those that do not.
__device__ __forceinline__ int tiles_of_sequence(int L, int nodes, const AttnParams &p) {
    return p.Hkv * tiles_per_head((L + KT - 1) / KT, nodes * p.G, p);
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

// Exclusive prefix sum of per-sequence tile counts into g_cum[0..B], the
// clamped prefix lengths into g_len[0..B) and the node counts into g_nn:
// wave 0 reads kv_len (and num_nodes) once per lane and scans with cross-lane
// shifts, one barrier for the whole workgroup.
template <int NT>
__device__ void build_cumulative(const AttnParams &p) {
    if (threadIdx.x < kWave) {
        const int lane = threadIdx.x;
        int carry = 0;
        for (int b0 = 0; b0 < p.B; b0 += kWave) {
            const int b = b0 + lane;
            const int L = b < p.B ? clamp_len(p.kv_len[b], p) : 0;
            const int nb = b < p.B ? nodes_of(b, p) : 0;
            const int t = b < p.B ? tiles_of_sequence(L, nb, p) : 0;
            int x = t;                                   // inclusive scan over the wave
            #pragma unroll
            for (int off = 1; off < kWave; off <<= 1) {
                const int y = __shfl_up(x, off);
                if (lane >= off) x += y;
            }
            if (b < p.B) {
                g_cum[b] = carry + x - t;
                g_len[b] = L;
                g_nn[b] = (unsigned short)nb;
            }
            carry += __shfl(x, kWave - 1);
        }
        if (lane == 0) g_cum[p.B] = carry;
    }
    __syncthreads();
}

// Piece set-up for pages shorter than a load block: page ids of pages
// [first, first + kPageCache) of sequence b (as far as it has them) into
// g_pages; all loads are issued before any is waited for.
template <int NT>
__device__ void load_pages(const AttnParams &p, int b, int first, int npages) {
    constexpr int PPT = (kPageCache + NT - 1) / NT;
    const int tid = threadIdx.x;
    const int n = min(kPageCache, npages - first);
    int pg[PPT];
    #pragma unroll
    for (int k = 0; k < PPT; ++k) {
        const int i = tid + k * NT;
        pg[k] = i < n ? p.page_table[(size_t)b * p.max_pages + first + i] : -1;
    }
    #pragma unroll
    for (int k = 0; k < PPT; ++k) {
        const int i = tid + k * NT;
        if (i < n) g_pages[i] = (pg[k] >= 0 && pg[k] < p.num_pages) ? pg[k] : -1;
    }
    __syncthreads();
}

// Ancestor sets of a tree of at most 64 nodes, by one wave and without
// barriers: lane i holds node i's set (one 64-bit word, reflexive) and the
// ancestor 2^k steps up; each round ORs in that ancestor's set and jumps
// twice as far (cross-lane reads see the values of the previous round), until
// no lane has an ancestor left. The caller's next workgroup barrier publishes
// g_anc.
// `pi` is node `lane`'s parent as loaded by the caller (any value for lanes >= N).
__device__ void build_ancestor_masks_wave(const AttnParams &p, int pi) {
    const int lane = threadIdx.x & (kWave - 1);
    int j = -1;
    if (lane < p.N) j = (pi < -1 || pi >= lane) ? -1 : pi;   // contract violation: treat as a root
    unsigned long long anc = lane < p.N ? (1ull << lane) : 0ull;
    while (__any(j >= 0)) {
        const int src = j >= 0 ? j : lane;
        const unsigned lo = (unsigned)__shfl((int)(unsigned)anc, src);
        const unsigned hi = (unsigned)__shfl((int)(unsigned)(anc >> 32), src);
        const int jj = __shfl(j, src);
        if (j >= 0) {
            anc |= ((unsigned long long)hi << 32) | lo;
            j = jj;
        }
    }
    if (lane < p.N) {
        g_anc[lane][0] = anc;
        g_anc[lane][1] = 0ull;
        g_anc[lane][2] = 0ull;
        g_anc[lane][3] = 0ull;
    }
}

// The same for up to kMaxNodes nodes, still one wave and no workgroup
// barrier: lane l owns nodes l, l + 64, ...; sets and jumps of the previous
// round are read from LDS (double buffered), and a wave-local wait for the
// LDS writes separates the rounds.
__device__ void build_ancestor_masks_wave_lds(const AttnParams &p, int b) {
    constexpr int K = kMaxNodes / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    int jmp[K];
    #pragma unroll
    for (int k = 0; k < K; ++k) {
        const int i = lane + k * kWave;
        jmp[k] = -1;
        if (i < p.N) {
            const int pi = p.parent[(size_t)b * p.N + i];
            jmp[k] = (pi < -1 || pi >= i) ? -1 : pi;
            #pragma unroll
            for (int w = 0; w < 4; ++w) g_anc[i][w] = (w == (i >> 6)) ? (1ull << (i & 63)) : 0ull;
            g_jump[0][i] = jmp[k];
        }
    }
    int cur = 0;
    for (;;) {
        bool more = false;
        #pragma unroll
        for (int k = 0; k < K; ++k) more |= jmp[k] >= 0;
        if (!__any(more)) break;
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        unsigned long long(*src)[4] = cur == 0 ? g_anc : g_anc_alt;
        unsigned long long(*dst)[4] = cur == 0 ? g_anc_alt : g_anc;
        #pragma unroll
        for (int k = 0; k < K; ++k) {
            const int i = lane + k * kWave;
            if (i >= p.N) continue;
            const int j = jmp[k];
            if (j >= 0) {
                #pragma unroll
                for (int w = 0; w < 4; ++w) dst[i][w] = src[i][w] | src[j][w];
                jmp[k] = g_jump[cur][j];
            } else {
                #pragma unroll
                for (int w = 0; w < 4; ++w) dst[i][w] = src[i][w];
            }
            g_jump[cur ^ 1][i] = jmp[k];
        }
        cur ^= 1;
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if (cur == 1) {
        #pragma unroll
        for (int k = 0; k < K; ++k) {
            const int i = lane + k * kWave;
            if (i < p.N)
                #pragma unroll
                for (int w = 0; w < 4; ++w) g_anc[i][w] = g_anc_alt[i][w];
        }
    }
}

template <int D, int NW, bool SMALL>
struct TileIssue {
    using Gm = Geo<D>;
    static constexpr int kLoadsPerWave = Gm::kBlocksPerTile / NW;   // per K (or V) tile
    static constexpr int LPT = kLoadsPerWave;
    static constexpr int KPB = Gm::kKeysPerBlock;     // keys per 1 KB load block
    static constexpr int C = Gm::kChunks;
    static_assert(LPT * NW == Gm::kBlocksPerTile, "blocks split evenly over waves");

    // Wave-uniform addresses of this wave's load blocks of one tile: the K and
    // V row of the block's first key, and how many of its KPB keys exist.
    struct Blocks {
        const char *k[LPT];
        const char *v[LPT];
        int nv[LPT];
    };

    int kib;                                          // this lane's key within a block
    unsigned row_off;                                 // kib * key row stride (bytes)
    unsigned chunk_off[LPT];                          // swizzled chunk offset per load
    unsigned lane_off[LPT];                           // i * KPB rows + row_off + chunk_off[i]
    // per unit
    const char *kc_g, *vc_g;                          // cache base + KV head g
    const char *kt_g, *vt_g;                          // tree row of node 0, KV head g
    unsigned row_bytes, page_bytes;                   // key row of all KV heads; one page
    int L, ntp, nodes;

    __device__ __forceinline__ void init(int wave_u, int lane, const AttnParams &p) {
        row_bytes = (unsigned)(p.Hkv * D * 2);
        page_bytes = row_bytes << p.p_shift;
        kib = lane / C;
        row_off = kib * row_bytes;
        #pragma unroll
        for (int i = 0; i < LPT; ++i) {
            const int kb = wave_u * LPT + i;
            chunk_off[i] = (unsigned)(((lane % C) ^ swz<C>((kb * KPB + kib) % C)) * 16);
            lane_off[i] = (unsigned)(i * KPB) * row_bytes + row_off + chunk_off[i];
        }
    }

    // Common case of a prefix tile: every row of the tile exists, this wave's
    // LPT blocks (consecutive keys) lie in one page, and that page id (pg0,
    // the page of the wave's first key) is valid. Then block i starts
    // i * KPB rows after `off`, the byte offset of the wave's first key row
    // from the cache base of KV head g. Returns false otherwise.
    __device__ __forceinline__ bool fast_offset(const AttnParams &p, int t, int wave_u, int pg0,
                                                unsigned long long &off) const {
        const int pos_w = t * KT + wave_u * LPT * KPB;
        if (LPT * KPB > p.P || t >= ntp || t * KT + KT > L || (unsigned)pg0 >= (unsigned)p.num_pages)
            return false;
        off = (unsigned long long)(unsigned)pg0 * page_bytes + (unsigned)(pos_w & (p.P - 1)) * row_bytes;
        return true;
    }

    // Direct-to-LDS loads of this wave's blocks of one K (or V) tile of the
    // common case (see fast_offset) into ring stage `stage`.
    __device__ __forceinline__ void issue_fast(unsigned long long off, bool is_v, int stage,
                                               int wave_u) const {
        unsigned char *dst = g_ring + stage * Gm::kStageBytes + (is_v ? Gm::kTileBytes : 0);
        const char *base = (is_v ? vc_g : kc_g) + off;
        #pragma unroll
        for (int i = 0; i < LPT; ++i)
            __builtin_amdgcn_global_load_lds((const GLOBAL_AS void *)(base + lane_off[i]),
                                             (LDS_AS void *)(dst + (wave_u * LPT + i) * 1024), 16, 0, 0);
    }

    __device__ __forceinline__ void set_unit(const AttnParams &p, int b, int g, int L_, int ntp_,
                                             int nodes_) {
        L = L_;
        ntp = ntp_;
        nodes = nodes_;
        kc_g = reinterpret_cast<const char *>(p.k_cache + (size_t)g * D);
        vc_g = reinterpret_cast<const char *>(p.v_cache + (size_t)g * D);
        kt_g = reinterpret_cast<const char *>(p.k_tree + ((size_t)b * p.N * p.Hkv + g) * D);
        vt_g = reinterpret_cast<const char *>(p.v_tree + ((size_t)b * p.N * p.Hkv + g) * D);
    }

    // Page ids of this wave's load blocks of prefix tile t, by scalar loads
    // through the constant address space: the ids land in SGPRs without
    // touching LDS. The index is clamped into the table row, so the load is
    // always in bounds; blocks() decides whether an id is used. Callers fetch
    // one tile period before the loads are issued, and nothing here waits for
    // the result.
    __device__ __forceinline__ void fetch_pages(const AttnParams &p, int b, int t, int wave_u,
                                                int (&pg)[LPT]) const {
        const CONST_AS int32_t *row =
            (const CONST_AS int32_t *)(p.page_table + (size_t)b * p.max_pages);
        #pragma unroll
        for (int i = 0; i < LPT; ++i) {
            const int pos0 = t * KT + (wave_u * LPT + i) * KPB;
            pg[i] = SMALL ? -1 : row[min(max(pos0 >> p.p_shift, 0), p.max_pages - 1)];
        }
    }

    // Block addresses of tile t. A block with no existing row (past the prefix,
    // past the sequence's nodes, or with an invalid page id) points at tree
    // node 0's row, which is always readable and finite; its rows are masked
    // later.
    __device__ __forceinline__ Blocks blocks(const AttnParams &p, int t, int wave_u,
                                             const int (&pg)[LPT]) const {
        Blocks r;
        if (t < ntp) {
            const bool full = t * KT + KT <= L;            // every row of the tile exists
            const int pos_w = t * KT + wave_u * LPT * KPB;  // first key of this wave's blocks
            #pragma unroll
            for (int i = 0; i < LPT; ++i) {
                const int pos0 = pos_w + i * KPB;
                const bool ok = (unsigned)pg[i] < (unsigned)p.num_pages && (full || pos0 < L);
                const size_t off = (size_t)(unsigned)pg[i] * page_bytes +
                                   (unsigned)((pos0 & (p.P - 1)) * row_bytes);
                r.k[i] = ok ? kc_g + off : kt_g;
                r.v[i] = ok ? vc_g + off : vt_g;
                r.nv[i] = !ok ? 0 : (full ? KPB : min(L - pos0, KPB));
            }
        } else {
            #pragma unroll
            for (int i = 0; i < LPT; ++i) {
                const int j0 = (t - ntp) * KT + (wave_u * LPT + i) * KPB;
                const int nv = min(max(nodes - j0, 0), KPB);
                const unsigned off = nv > 0 ? (unsigned)j0 * (unsigned)row_bytes : 0u;
                r.k[i] = kt_g + off;
                r.v[i] = vt_g + off;
                r.nv[i] = nv;
            }
        }
        return r;
    }

    // Direct-to-LDS loads of this wave's blocks of one K (or V) tile into ring
    // stage `stage`.
    __device__ __forceinline__ void issue(const Blocks &bl, bool is_v, int stage, int wave_u) const {
        unsigned char *dst = g_ring + stage * Gm::kStageBytes + (is_v ? Gm::kTileBytes : 0);
        #pragma unroll
        for (int i = 0; i < LPT; ++i) {
            const char *addr = (is_v ? bl.v[i] : bl.k[i]) + ((kib < bl.nv[i] ? row_off : 0u) + chunk_off[i]);
            __builtin_amdgcn_global_load_lds((const GLOBAL_AS void *)addr,
                                             (LDS_AS void *)(dst + (wave_u * LPT + i) * 1024), 16, 0, 0);
        }
    }

    // Pages shorter than a load block: every lane looks up its own page in the
    // LDS page-id window (prefix tiles only).
    __device__ __forceinline__ void issue_small(const AttnParams &p, int t, bool is_v, int page_first,
                                                int wave_u) const {
        unsigned char *dst = g_ring + (t & (NS - 1)) * Gm::kStageBytes + (is_v ? Gm::kTileBytes : 0);
        #pragma unroll
        for (int i = 0; i < LPT; ++i) {
            const int pos = t * KT + (wave_u * LPT + i) * KPB + kib;
            const char *row = is_v ? vt_g : kt_g;
            if (pos < L) {
                const int id = g_pages[(pos >> p.p_shift) - page_first];
                if (id >= 0)
                    row = (is_v ? vc_g : kc_g) + (size_t)(unsigned)id * page_bytes + (size_t)(pos & (p.P - 1)) * row_bytes;
            }
            __builtin_amdgcn_global_load_lds((const GLOBAL_AS void *)(row + chunk_off[i]),
                                             (LDS_AS void *)(dst + (wave_u * LPT + i) * 1024), 16, 0, 0);
        }
    }
};

// Wait until at most n of this wave's vector-memory operations are still in
// flight; a count without its own case waits for the next smaller one.
__device__ __forceinline__ void wait_vm_at_most(int n) {
    if (n >= 63) wait_vmcnt<63>();
    else if (n >= 48) wait_vmcnt<48>();
    else if (n >= 32) wait_vmcnt<32>();
    else if (n >= 24) wait_vmcnt<24>();
    else if (n >= 16) wait_vmcnt<16>();
    else if (n >= 12) wait_vmcnt<12>();
    else if (n >= 8) wait_vmcnt<8>();
    else if (n >= 6) wait_vmcnt<6>();
    else if (n >= 4) wait_vmcnt<4>();
    else if (n >= 2) wait_vmcnt<2>();
    else if (n >= 1) wait_vmcnt<1>();
    else wait_vmcnt<0>();
}

// LDS-read wait with a count that is a constant once the caller is unrolled.
__device__ __forceinline__ void lds_wait_n(int n) {
    switch (n) {
        case 0: lds_wait<0>(); break;
        case 1: lds_wait<1>(); break;
        case 2: lds_wait<2>(); break;
        case 3: lds_wait<3>(); break;
        case 4: lds_wait<4>(); break;
        case 5: lds_wait<5>(); break;
        case 6: lds_wait<6>(); break;
        case 7: lds_wait<7>(); break;
        case 8: lds_wait<8>(); break;
        default: lds_wait<0>(); break;
    }
}

// Per-wave state of one piece: Q fragments (MFMA B operand), O^T
// accumulators, the probabilities of the tile whose PV product is pending,
// running max and sum.
template <int D>
struct WaveState {
    static constexpr int NKS = D / 16;     // MFMA k-steps over the head dim
    static constexpr int NDT = D / 32;     // 32-wide head-dim tiles of the output
    bf16x8 qf[NKS];
    f32x16 o[NDT];
    u32x4 pb[4];                           // P^T as bf16 pairs, 16 keys per k-step
    float m_run;                           // running max (raw score units)
    float msc;                             // m_run * scale_log2 (0 while m_run is -inf)
    float l_run;                           // this lane's part of the running sum
};

// Visible keys of tile j for the lane's row: every key of a full prefix tile
// (masked = false, wave-uniform), the keys below the prefix length on the last
// prefix tile, the node's ancestors on a tree tile. Bit k of (vis_hi:vis_lo)
// is the key the lane holds at position k of a half-0 lane (the lane's own
// half already shifted in).
struct TileMask {
    bool masked;
    unsigned vis_lo, vis_hi;
};

// Key position (within the tile) of accumulator element r of half hf, for a
// lane of half 0; a lane of half 1 holds the key 4 positions later.
__host__ __device__ constexpr int key_of(int hf, int r) { return hf * 32 + (r >> 2) * 8 + (r & 3); }

// Exponentials of 2 scores of one tile into a bf16 pair of P^T and the
// running sum: x = 2^(s * c - msc).
// The results are tied (empty volatile asm) so that the computation stays in
// the MFMA slot it was written in instead of sinking to its first use.
__device__ __forceinline__ unsigned exp_pair(float s0, float s1, float c, float msc, float &sum) {
    const float x0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s0, c, -msc));
    const float x1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s1, c, -msc));
    sum += x0 + x1;
    const bf16x2 pr = {(__bf16)x0, (__bf16)x1};
    unsigned u = __builtin_bit_cast(unsigned, pr);
    tie(u);
    tie(sum);
    return u;
}

// One tile period of one wave.
//   CUR:  part A computes tile j's scores S^T = K_j Q^T into s0 (keys 0..31)
//         and s1 (keys 32..63); part B masks them, takes their maximum,
//         decides the running maximum and exponentiates half 0 into P^T.
//   PREV: the first half of part A exponentiates the previous tile's half 1
//         (in s1, consumed before this tile's half-1 products overwrite it);
//         part B adds P^T V_{j-1} to O.
// The VALU slices sit between the MFMAs of their part, so the matrix pipe and
// the VALU of one wave overlap; two 16-register score halves are alive at any
// time. LDS operand reads run two MFMAs ahead with explicit waits.
template <int D, bool PREV, bool CUR>
__device__ __forceinline__ void tile_period(WaveState<D> &st, f32x16 &sc0, f32x16 &sc1,
                                            unsigned kaddr, unsigned vaddr, const TileMask &mk,
                                            float c) {
    f32x16 *sc[2] = {&sc0, &sc1};
    using Gm = Geo<D>;
    constexpr int NKS = D / 16, NDT = D / 32;
    constexpr int C = Gm::kChunks;
    constexpr int SA = 2 * NKS;            // part A slots: one S MFMA each
    constexpr int SB = 4 * NDT;            // part B slots: one PV MFMA each
    constexpr int NSLOT = SA + SB;
    constexpr int R = 2;                   // operand reads run this many slots ahead
    constexpr int PPA = 8 / NKS;                       // half-1 pairs per slot of part A's first half
    // first part-B slot of the half-0 pairs: after the decision (slot 5) and
    // after the PV MFMAs that read P^T k-steps 0 and 1 have issued
    constexpr int B0 = 2 * NDT > 6 ? 2 * NDT : 6;
    constexpr int PPB = (8 + (SB - B0) - 1) / (SB - B0);   // half-0 pairs per part-B slot
    static_assert(NKS <= 8 && 8 % NKS == 0 && SB > B0, "slice shapes");
    auto active = [](int s) { return s < SA ? CUR : PREV; };
    auto ops = [&](int s) { return (s < NSLOT && active(s)) ? (s < SA ? 1 : 2) : 0; };
    u32x4 kb[SA];
    u32x2 vb[SB][2];
    auto issue_reads = [&](int s) {
        if (s >= NSLOT || !active(s)) return;
        if (s < SA) {
            const int hf = s / NKS, ks = s % NKS;
            asm volatile("ds_read_b128 %0, %1 offset:%2"
                         : "=v"(kb[s])
                         : "v"(kaddr ^ ((unsigned)ks << 5)), "i"(hf * 32 * Gm::kRowBytes));
        } else {
            const int b = s - SA, kk = b / NDT, dt = b % NDT;
            #pragma unroll
            for (int rr = 0; rr < 2; ++rr) {
                const unsigned flip = (unsigned)((dt * 4) ^ swz<C>((rr * 8) % C)) << 4;
                asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2"
                             : "=v"(vb[b][rr])
                             : "v"(vaddr ^ flip), "i"((kk * 16 + rr * 8) * Gm::kRowBytes));
            }
        }
    };
    float psa = 0.f, psb = 0.f;
    float m8[4];
    float alpha = 1.f;
    bool any_raise = false;
    #pragma unroll
    for (int s = 0; s < R; ++s) issue_reads(s);
    #pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
        issue_reads(s + R);
        if (active(s)) {
            int newer = 0;
            #pragma unroll
            for (int k = 1; k <= R; ++k) newer += ops(s + k);
            lds_wait_n(newer);
            if (s < SA) {
                const int hf = s / NKS, ks = s % NKS;
                tie(kb[s]);
                const f32x16 acc = ks == 0 ? f32x16{} : *sc[hf];   // a chain starts from zero
                *sc[hf] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kb[s]),
                                                                  st.qf[ks], acc, 0, 0, 0);
            } else {
                const int b = s - SA, kk = b / NDT, dt = b % NDT;
                tie(vb[b][0]);
                tie(vb[b][1]);
                const u32x4 a = {vb[b][0][0], vb[b][0][1], vb[b][1][0], vb[b][1][1]};
                st.o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, st.pb[kk]), st.o[dt],
                    0, 0, 0);
            }
        }
        if (PREV && s < NKS) {
            // pairs of the previous tile's half 1 (keys 32 + 2i, 33 + 2i: P^T
            // k-steps 2, 3), all before slot NKS overwrites s1
            #pragma unroll
            for (int u = 0; u < PPA; ++u) {
                const int i = s * PPA + u, kk = 2 + (i >> 2), w = i & 3;
                st.pb[kk][w] = exp_pair(sc1[2 * i], sc1[2 * i + 1], c, st.msc, psa);
            }
        }
        if (PREV && s == NKS - 1) st.l_run += psa;
        if (CUR && s == SA + 1 && mk.masked) {
            // the last prefix tile or a tree tile: invisible keys become -inf
            // (selected, never added), in place
            #pragma unroll
            for (int hf = 0; hf < 2; ++hf)
                #pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int k = key_of(hf, r);
                    const unsigned word = k < 32 ? mk.vis_lo : mk.vis_hi;
                    (*sc[hf])[r] = ((word >> (k & 31)) & 1u) ? (*sc[hf])[r] : kNegInf;
                }
        }
        if (CUR && s >= SA + 1 && s < SA + 5) {
            // maximum of 8 of this tile's scores (chunk q: half q / 2, elements
            // 8 (q % 2) .. +8)
            const int q = s - SA - 1, hf = q >> 1, r0 = (q & 1) * 8;
            const f32x16 &v = *sc[hf];
            const float a = max3(v[r0], v[r0 + 1], v[r0 + 2]);
            const float b = max3(v[r0 + 3], v[r0 + 4], v[r0 + 5]);
            m8[q] = max3(a, b, max3(v[r0 + 6], v[r0 + 7], v[r0 + 7]));
            tie(m8[q]);
        }
        if (CUR && s == SA + 5) {
            // The running max is only raised when a score exceeds it by more
            // than kRescaleSlack (log2 units), so O is rarely rescaled. The
            // sum is rescaled here; O after this period's PV products.
            const float tmax = halves_max(max3(m8[0], m8[1], max3(m8[2], m8[3], m8[3])));
            const bool raise = tmax * c > st.m_run * c + kRescaleSlack;
            any_raise = __any(raise);
            if (any_raise) {
                const float m_new = raise ? tmax : st.m_run;
                alpha = (st.m_run == kNegInf) ? 0.f
                        : __builtin_amdgcn_exp2f((st.m_run - m_new) * c);
                st.l_run *= alpha;
                st.m_run = m_new;
            }
            st.msc = (st.m_run == kNegInf) ? 0.f : st.m_run * c;
        }
        if (CUR && s >= SA + B0) {
            #pragma unroll
            for (int u = 0; u < PPB; ++u) {
                const int i = (s - SA - B0) * PPB + u;     // pair i of half 0: keys 2i, 2i + 1
                if (i < 8) st.pb[i >> 2][i & 3] = exp_pair(sc0[2 * i], sc0[2 * i + 1], c, st.msc, psb);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    if (CUR) {
        st.l_run += psb;
        if (any_raise) {
            #pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
                #pragma unroll
                for (int r = 0; r < 16; ++r) st.o[dt][r] *= alpha;
        }
    }
}

// ---- units of at most 16 query rows (the paper's own MHA shape: 12 nodes x 1
// head per KV head). Every row tile of the main scheme would be mostly empty,
// so here the workgroup's waves take the unit's tiles in turn (tile j belongs
// to wave j mod NW) and compute it whole with v_mfma_f32_16x16x32_bf16: keys on
// M (16 per block, 4 blocks per tile), the 16 rows on N, head dim on K. Lane l
// holds row l % 16; in a 16x16 accumulator it holds entries m = 4 (l / 16) + i,
// i < 4, so S gives it keys 16 kb + 4 (l / 16) + i of every key block kb. The
// PV product takes P^T straight from there: its k-step over key blocks (kb0,
// kb1) pairs k = 8 (l / 16) + i with key 16 kb0 + 4 (l / 16) + i and
// k = 8 (l / 16) + 4 + i with key 16 kb1 + 4 (l / 16) + i, and the V^T operand
// is read with the same key order through ds_read_b64_tr_b16 (a 16-lane group
// reads 4 key rows x 16 head-dim columns; lane i of the group receives column
// i of the 4 rows). Each wave keeps its own running max, sum and O^T for its
// tiles; the waves' states are combined with the log-sum-exp rule at the end
// of the piece. Tile loads stay cooperative (all waves, one barrier per tile),
// and with one wave computing per tile the period is bound by the loads.
template <int D>
struct NarrowState {
    static constexpr int NKS = D / 32;     // k-steps over the head dim (S)
    static constexpr int NDB = D / 16;     // 16-wide head-dim blocks of O^T
    bf16x8 qf[NKS];
    f32x4 o[NDB];
    float m_run, msc, l_run;
};

// Tile j for the owning wave. kaddr/vaddr: the stage's K and V tile bases (LDS
// byte addresses); vis: the visible keys of the lane's row (bit = key in tile),
// all ones for a full prefix tile.
template <int D>
__device__ __forceinline__ void narrow_tile(NarrowState<D> &st, unsigned kbase, unsigned vbase,
                                            bool masked, unsigned long long vis, float c, int lane) {
    using Gm = Geo<D>;
    constexpr int C = Gm::kChunks;
    constexpr int NKS = D / 32, NDB = D / 16;
    const int g = lane >> 4, i16 = lane & 15;
    // S^T blocks; the K reads of block kb + 1 are in flight during block kb's MFMAs
    f32x4 sb[4];
    u32x4 a[2][NKS];
    auto read_k = [&](int kb, u32x4 (&dst)[NKS]) {
        const int key = kb * 16 + i16;
        const unsigned row = kbase + key * Gm::kRowBytes;
        #pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
            asm volatile("ds_read_b128 %0, %1" : "=v"(dst[ks])
                         : "v"(row + ((unsigned)((4 * ks + g) ^ swz<C>(key % C)) << 4)));
    };
    read_k(0, a[0]);
    #pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
        if (kb + 1 < 4) {
            read_k(kb + 1, a[(kb + 1) & 1]);
            lds_wait<NKS>();
        } else {
            lds_wait<0>();
        }
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        #pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
            tie(a[kb & 1][ks]);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[kb & 1][ks]),
                                                          st.qf[ks], acc, 0, 0, 0);
        }
        sb[kb] = acc;
    }
    if (masked) {
        #pragma unroll
        for (int kb = 0; kb < 4; ++kb)
            #pragma unroll
            for (int i = 0; i < 4; ++i)
                sb[kb][i] = ((vis >> (kb * 16 + 4 * g + i)) & 1ull) ? sb[kb][i] : kNegInf;
    }
    float mt = kNegInf;
    #pragma unroll
    for (int kb = 0; kb < 4; ++kb) mt = fmaxf(mt, fmaxf(fmaxf(sb[kb][0], sb[kb][1]), fmaxf(sb[kb][2], sb[kb][3])));
    mt = rows_max(mt);
    const bool raise = mt * c > st.m_run * c + kRescaleSlack;
    if (__any(raise)) {
        const float m_new = raise ? mt : st.m_run;
        const float alpha = (st.m_run == kNegInf) ? 0.f : __builtin_amdgcn_exp2f((st.m_run - m_new) * c);
        st.l_run *= alpha;
        #pragma unroll
        for (int db = 0; db < NDB; ++db)
            #pragma unroll
            for (int i = 0; i < 4; ++i) st.o[db][i] *= alpha;
        st.m_run = m_new;
    }
    st.msc = (st.m_run == kNegInf) ? 0.f : st.m_run * c;
    bf16x8 pb[2];
    float ps = 0.f;
    #pragma unroll
    for (int kb = 0; kb < 4; ++kb)
        #pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float x = __builtin_amdgcn_exp2f(__builtin_fmaf(sb[kb][i], c, -st.msc));
            ps += x;
            pb[kb >> 1][(kb & 1) * 4 + i] = (__bf16)x;
        }
    st.l_run += ps;
    // O^T += V^T P^T, two k-steps of 32 keys; step q = kst * NDB + db, its two
    // transposing reads issued two steps ahead
    constexpr int NQ = 2 * NDB;
    u32x2 v[NQ][2];
    auto read_v = [&](int q) {
        const int kst = q / NDB, db = q % NDB;
        #pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int key = (2 * kst + r) * 16 + 4 * g + (i16 >> 2);
            const int chunk = 2 * db + ((i16 & 3) >> 1);
            const unsigned addr = vbase + key * Gm::kRowBytes +
                                  ((unsigned)(chunk ^ swz<C>(key % C)) << 4) + (i16 & 1) * 8;
            asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v[q][r]) : "v"(addr));
        }
    };
    read_v(0);
    read_v(1);
    #pragma unroll
    for (int q = 0; q < NQ; ++q) {
        if (q + 2 < NQ) {
            read_v(q + 2);
            lds_wait<4>();
        } else if (q + 1 < NQ) {
            lds_wait<2>();
        } else {
            lds_wait<0>();
        }
        tie(v[q][0]);
        tie(v[q][1]);
        const int kst = q / NDB, db = q % NDB;
        const u32x4 av = {v[q][0][0], v[q][0][1], v[q][1][0], v[q][1][1]};
        st.o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av), pb[kst],
                                                           st.o[db], 0, 0, 0);
    }
}

template <int D, int NW, bool SMALL, bool NARROW>
__global__ __launch_bounds__(NW * kWave) void tree_attention_kernel(AttnParams p) {
    using Gm = Geo<D>;
    using Issue = TileIssue<D, NW, SMALL>;
    constexpr int NT = NW * kWave;
    constexpr int NKS = D / 16;
    constexpr int NDT = D / 32;
    constexpr int LPT = Issue::kLoadsPerWave;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave_u = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int half = lane >> 5;
    const int col = lane & 31;
    const int w = xcd_contiguous_id(blockIdx.x, p.num_wg);

    build_cumulative<NT>(p);

    const int total = g_cum[p.B];
    // Workgroup u < nw takes virtual tiles [share_start(u), share_start(u + 1)):
    // shares differ by at most one tile and none is empty (nw <= total), so the
    // pieces of a split unit sit in consecutive workgroups. Workgroups past nw
    // (only when the length hint overstated the work) have nothing to do.
    const int nw = min(p.num_wg, total);
    auto share_start = [&](int u) { return (int)(((long long)min(u, nw) * total) / max(nw, 1)); };
    auto share_of = [&](int t) { return (int)(((long long)(t + 1) * nw - 1) / total); };
    const int start = share_start(w);
    const int end = share_start(w + 1);
    const unsigned ring_base = lds_addr(g_ring);
    Issue ld;
    ld.init(wave_u, lane, p);

    // lane-constant parts of the LDS fragment addresses (see swz)
    const unsigned k_lane = col * Gm::kRowBytes + ((half ^ swz<Gm::kChunks>(col % Gm::kChunks)) << 4);
    const int va = ((lane >> 4) & 1) * 2 + ((lane & 3) >> 1);
    const int vb = half * 4 + ((lane & 15) >> 2);
    const unsigned v_lane = vb * Gm::kRowBytes + ((va ^ swz<Gm::kChunks>(vb)) << 4) + (lane & 1) * 8;

    int pos = start;
    int anc_b = -1;                 // sequence whose ancestor sets are in g_anc
    if (start >= end && tid == 0) p.ws_desc[w * 4] = -1;
    while (pos < end) {
        // ---- locate the unit holding tile `pos`
        int lo = 0, hi = p.B - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (g_cum[mid] <= pos) lo = mid; else hi = mid - 1;
        }
        const int b = lo;
        const int L = g_len[b];
        const int nodes = g_nn[b];
        const int rows_b = nodes * p.G;                 // this sequence's query rows per KV head
        const int ntp = (L + KT - 1) / KT;
        const int C = p.setup_tiles;
        const int per_g = tiles_per_head(ntp, rows_b, p);
        int off = pos - g_cum[b];
        const int g = off / per_g;
        off -= g * per_g;
        int rb = 0;
        int ulen = ntp + tree_tiles_of_block(0, rows_b, p);     // real tiles of the unit
        while (off >= C + ulen) {
            off -= C + ulen;
            ++rb;
            ulen = ntp + tree_tiles_of_block(rb, rows_b, p);
        }
        // this share covers virtual tiles [off, v_end) of the unit; real tile
        // r is virtual tile C + r
        const int v_end = min(C + ulen, off + (end - pos));
        const int unit_real_start = pos - off + C;    // share coordinate of real tile 0
        const int t0 = max(off - C, 0);
        // Page ids of the first four tiles (scalar loads): for narrow units first
        // of all, so that their latency overlaps the rest of the set-up; for the
        // others after the parent links (holding them that long costs the
        // eight-wave kernel spills). Later sub-ranges fetch their own.
        int ids[4][Issue::kLoadsPerWave];
        if constexpr (NARROW) {
            #pragma unroll
            for (int i = 0; i < 4; ++i) ld.fetch_pages(p, b, t0 + i, wave_u, ids[i]);
        }
        if (pos == start && tid == 0) {
            // the merge kernel's entry for this workgroup: the split unit whose
            // last piece is this share's first, if any
            const int wf = share_of(unit_real_start);
            const bool mine = unit_real_start < start && share_of(unit_real_start + ulen - 1) == w;
            *reinterpret_cast<i32x4 *>(p.ws_desc + w * 4) =
                mine ? i32x4{b, g, rb | (nodes << 8), wf * 2 + (unit_real_start <= share_start(wf) ? 0 : 1)}
                     : i32x4{-1, 0, 0, 0};
        }
        pos += v_end - off;
        const int t_end = v_end - C;
        if (t_end <= t0) continue;                    // only set-up tiles of this unit
        const bool complete = (t0 == 0 && t_end == ulen);

        // Parent links for the ancestor sets (trees of up to 64 nodes), loaded
        // before any other load of the piece so that waiting for them never
        // waits for the tile loads behind them.
        const bool has_tree = t_end > ntp;
        const bool need_anc = has_tree && anc_b != b;
        int par_pre = -1;
        if (need_anc && wave_u == 0 && p.N <= kWave && lane < p.N)
            par_pre = p.parent[(size_t)b * p.N + lane];
        if constexpr (!NARROW) {
            #pragma unroll
            for (int i = 0; i < 4; ++i) ld.fetch_pages(p, b, t0 + i, wave_u, ids[i]);
        }

        // ---- this wave's 32 query rows: Q fragments stay in registers. A row
        // past the unit's last one loads the unit's first row instead (rows are
        // independent through both products and the softmax, and such rows are
        // never stored), so the loads need no branch and nothing waits for them
        // before the first score product.
        const int row = rb * p.rows_per_block + wave_u * kRowsPerWave + col;
        const bool row_ok = row < rows_b;
        const int qrow = row_ok ? row : rb * p.rows_per_block;
        const int node = qrow / p.G;
        const int hq = g * p.G + qrow % p.G;
        WaveState<D> st;
        NarrowState<D> ns;
        // narrow units: lane l holds row l % 16 (rows past the unit's last load
        // its first row, never stored) and head-dim columns 8 (l / 16) + 32 ks
        const int nrow = NARROW ? min(lane & 15, rows_b - 1) : 0;
        const int nnode = nrow / p.G;
        if constexpr (!NARROW) {
            const uint16_t *qp = p.q + (((size_t)b * p.N + node) * p.Hq + hq) * D + half * 8;
            #pragma unroll
            for (int ks = 0; ks < NKS; ++ks)
                st.qf[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8 *>(qp + ks * 16));
            #pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
                #pragma unroll
                for (int r = 0; r < 16; ++r) st.o[dt][r] = 0.f;
            st.m_run = kNegInf;
            st.msc = 0.f;
            st.l_run = 0.f;
        } else {
            const int nhq = g * p.G + nrow % p.G;
            const uint16_t *qp = p.q + (((size_t)b * p.N + nnode) * p.Hq + nhq) * D + (lane >> 4) * 8;
            #pragma unroll
            for (int ks = 0; ks < D / 32; ++ks)
                ns.qf[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8 *>(qp + ks * 32));
            #pragma unroll
            for (int db = 0; db < D / 16; ++db) ns.o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
            ns.m_run = kNegInf;
            ns.msc = 0.f;
            ns.l_run = 0.f;
        }

        const int npages = (L + p.P - 1) >> p.p_shift;
        auto kaddr_of = [&](int t) { return ring_base + (t & (NS - 1)) * Gm::kStageBytes + k_lane; };
        auto vaddr_of = [&](int t) {
            return ring_base + (t & (NS - 1)) * Gm::kStageBytes + Gm::kTileBytes + v_lane;
        };
        // Scores of the current tile: half 0 in s0, half 1 in s1 (exponentiated
        // early in the next period).
        f32x16 s0, s1;

        // The segment runs in sub-ranges whose prefix pages fit the LDS page-id
        // window (one sub-range unless a piece spans more than kPageCache pages).
        for (int ta = t0; ta < t_end;) {
            const int page_first = (ta * KT) >> p.p_shift;
            int tb = t_end;
            if (ta < ntp) {
                const int t_cov = ((page_first + kPageCache) << p.p_shift) / KT;   // first tile not covered
                if (t_cov < ntp) tb = min(tb, t_cov);
            }
            const bool first = (ta == t0);
            // page ids in LDS only for pages shorter than a load block; ancestor
            // sets only when this piece reaches the tree tiles and the workgroup
            // has not built them for this sequence already
            const bool want_anc = first && need_anc;
            if (SMALL && ta < ntp) load_pages<NT>(p, b, page_first, npages);

            const int T = tb - ta;
            // Tile i of the sub-range (K and V of tile ta + i) goes to ring stage
            // (ta + i) % NS. Period j computes S with K_j and PV with V_{j-1}, and
            // issues K_{j+3} and V_{j+2}: the K half it refills last held K_{j-1}
            // (read in period j - 1), the V half V_{j-2} (read in period j - 1),
            // both before the barrier that opens period j. Every load is issued
            // about three periods before it is read.
            int pk[LPT];                       // page ids of the next K tile to be loaded
            typename Issue::Blocks bk;         // block addresses of the last K tile issued,
            bool fast = false;                 // or, when `fast`, its common-case offset
            unsigned long long foff = 0;
            auto blocks_of = [&](int i) { return ld.blocks(p, ta + i, wave_u, pk); };
            auto issue_half = [&](int i, bool is_v, const typename Issue::Blocks &bl) {
                const int t = ta + i;
                if (SMALL && t < ntp) ld.issue_small(p, t, is_v, page_first, wave_u);
                else ld.issue(bl, is_v, t & (NS - 1), wave_u);
            };
            ld.set_unit(p, b, g, L, ntp, nodes);
            {
                // narrow units: full prefix tiles take the fast address path here too
                typename Issue::Blocks b0, b1;
                unsigned long long f0 = 0, f1 = 0;
                const bool fa0 = NARROW && !SMALL && ld.fast_offset(p, ta, wave_u, ids[0][0], f0);
                const bool fa1 = NARROW && !SMALL && T > 1 && ld.fast_offset(p, ta + 1, wave_u, ids[1][0], f1);
                fast = NARROW && !SMALL && T > 2 && ld.fast_offset(p, ta + 2, wave_u, ids[2][0], foff);
                if (!fa0) {
                    #pragma unroll
                    for (int k = 0; k < LPT; ++k) pk[k] = ids[0][k];
                    b0 = blocks_of(0);
                }
                if (T > 1 && !fa1) {
                    #pragma unroll
                    for (int k = 0; k < LPT; ++k) pk[k] = ids[1][k];
                    b1 = blocks_of(1);
                }
                if (T > 2 && !fast) {
                    #pragma unroll
                    for (int k = 0; k < LPT; ++k) pk[k] = ids[2][k];
                    bk = blocks_of(2);         // K_2 now, V_2 in period 0 (narrow: now)
                }
                auto issue_pro = [&](int i, bool is_v, bool fa, unsigned long long fo,
                                     const typename Issue::Blocks &bl) {
                    if (fa) ld.issue_fast(fo, is_v, (ta + i) & (NS - 1), wave_u);
                    else issue_half(i, is_v, bl);
                };
                // issue order K_0, V_0, K_1, V_1, K_2 (, V_2) (the waits below count on it)
                issue_pro(0, false, fa0, f0, b0);
                issue_pro(0, true, fa0, f0, b0);
                if (T > 1) {
                    issue_pro(1, false, fa1, f1, b1);
                    issue_pro(1, true, fa1, f1, b1);
                }
                if (T > 2) issue_pro(2, false, fast, foff, bk);
                if (NARROW && T > 2) issue_pro(2, true, fast, foff, bk);
                #pragma unroll
                for (int k = 0; k < LPT; ++k) pk[k] = ids[3][k];
            }
            // Ancestor sets, while the first loads are in flight, by one wave (the
            // others read them only after the next workgroup barrier): in
            // registers up to 64 nodes, else in LDS.
            if (want_anc) {
                if (wave_u == 0) {
                    tie(par_pre);              // first use here, behind the tile loads
                    if (p.N <= kWave) build_ancestor_masks_wave(p, par_pre);
                    else build_ancestor_masks_wave_lds(p, b);
                }
                anc_b = b;
            }

            // Loads this wave issues at the end of period i (V_{i+2}, K_{i+3} when they exist).
            auto loads_in = [&](int i) { return (i + 3 < T ? LPT : 0) + (i + 2 < T ? LPT : 0); };
            // Opening of period j: K_j and V_{j-1} have landed for every wave (this
            // wave's later loads may still be in flight) and every wave is done
            // with period j - 1; then tile j's mask.
            TileMask mk;
            unsigned long long nvis = ~0ull;   // narrow units: the visible keys of the lane's row
            auto open_period = [&](int j) {
                int newer;                     // loads issued after the last one period j needs
                if (NARROW) newer = 2 * LPT * ((j + 1 < T ? 1 : 0) + (j + 2 < T ? 1 : 0));   // tiles j+1, j+2
                else if (j == 0) newer = LPT * ((T > 1 ? 2 : 0) + (T > 2 ? 1 : 0)) + LPT;   // V_0, K_1, V_1, K_2
                else if (j == 1) newer = LPT * ((T > 1 ? 1 : 0) + (T > 2 ? 1 : 0)) + loads_in(0);
                else if (j == 2) newer = loads_in(0) + loads_in(1);
                else newer = loads_in(j - 2) + loads_in(j - 1);
                wait_vm_at_most(newer);
                lds_barrier();
                const int t = ta + j;
                unsigned long long vis;
                if (t < ntp) {
                    const int lim_t = L - t * KT;      // keys at or past it lie beyond the prefix
                    mk.masked = lim_t < KT;
                    vis = lim_t >= KT ? ~0ull : ((1ull << lim_t) - 1ull);
                } else {
                    mk.masked = true;
                    vis = g_anc[NARROW ? nnode : node][t - ntp];
                }
                nvis = vis;
                vis >>= half * 4;
                mk.vis_lo = (unsigned)vis;
                mk.vis_hi = (unsigned)(vis >> 32);
            };
            // End of period j: this wave's loads of K_{j+3} and V_{j+2}, all at
            // once. (LDS-DMA writes slow down the LDS operand reads of every wave
            // of the CU; one burst per period costs far less than loads spread
            // between the MFMAs.) The K half they refill last held K_{j-1}, the V
            // half V_{j-2}, both read before the barrier that opened period j.
            // Then the page ids of K_{j+4}, by scalar loads that complete by the
            // next barrier.
            auto close_period = [&](int j) {
                if (j + 2 < T) {                   // V_{j+2}: the addresses of K_{j+2}
                    if (fast) ld.issue_fast(foff, true, (ta + j + 2) & (NS - 1), wave_u);
                    else issue_half(j + 2, true, bk);
                }
                if (j + 3 < T) {
                    fast = !SMALL && ld.fast_offset(p, ta + j + 3, wave_u, pk[0], foff);
                    if (fast) {
                        ld.issue_fast(foff, false, (ta + j + 3) & (NS - 1), wave_u);
                    } else {
                        if (!(SMALL && ta + j + 3 < ntp)) bk = blocks_of(j + 3);
                        issue_half(j + 3, false, bk);
                    }
                }
                ld.fetch_pages(p, b, ta + j + 4, wave_u, pk);
            };
            int j = 0;
            auto run = [&](auto prev, auto cur) {
                constexpr bool P_ = decltype(prev)::value, C_ = decltype(cur)::value;
                const int jj = j;
                tile_period<D, P_, C_>(st, s0, s1, C_ ? kaddr_of(ta + jj) : 0u,
                                       P_ ? vaddr_of(ta + jj - 1) : 0u, mk, p.scale_log2);
                if (C_) close_period(jj);
            };
            // Before the last PV: V of the last tile has landed for every wave.
            auto close_periods = [&]() {
                wait_vm_at_most(0);
                lds_barrier();
            };
            using T_ = std::true_type;
            using F_ = std::false_type;
            if constexpr (NARROW) {
                // tile t is computed whole by wave t % NW (= its ring stage); at
                // the end of period j every wave issues its share of tile j + 3
                // (K and V), whose stage last held tile j - 1, computed in period
                // j - 1, before the barrier that opened period j
                for (j = 0; j < T; ++j) {
                    open_period(j);
                    const int t = ta + j;
                    if ((t & (NS - 1)) == wave_u)
                        narrow_tile<D>(ns, ring_base + (t & (NS - 1)) * Gm::kStageBytes,
                                       ring_base + (t & (NS - 1)) * Gm::kStageBytes + Gm::kTileBytes,
                                       mk.masked, nvis, p.scale_log2, lane);
                    if (j + 3 < T) {
                        fast = !SMALL && ld.fast_offset(p, t + 3, wave_u, pk[0], foff);
                        if (fast) {
                            ld.issue_fast(foff, false, (t + 3) & (NS - 1), wave_u);
                            ld.issue_fast(foff, true, (t + 3) & (NS - 1), wave_u);
                        } else {
                            if (!(SMALL && t + 3 < ntp)) bk = blocks_of(j + 3);
                            issue_half(j + 3, false, bk);
                            issue_half(j + 3, true, bk);
                        }
                    }
                    ld.fetch_pages(p, b, t + 4, wave_u, pk);
                }
            } else {
                open_period(0);
                run(F_{}, T_{});
                for (j = 1; j < T; ++j) {
                    open_period(j);
                    run(T_{}, T_{});
                }
                close_periods();
                run(T_{}, F_{});               // PV of the last tile
            }
            ta = tb;
            if (ta < t_end) {
                #pragma unroll
                for (int i = 0; i < 4; ++i) ld.fetch_pages(p, b, ta + i, wave_u, ids[i]);
            }
            __syncthreads();               // ring and page ids are reused next
        }

        // ---- finish the segment
        // The normalised rows leave through this wave's slice of the (now idle)
        // LDS ring, transposed there so that every global store writes whole
        // rows (16 lanes x 16 bytes per 256-byte row) instead of 8-byte pieces
        // of 32 rows. A complete unit writes out and lse; a piece of a split
        // unit writes its output normalised by its own sum (bf16) and its (max,
        // sum) pair (fp32): slot 0 holds the piece that continues a unit from
        // before this share, slot 1 the one that starts inside it.
        const int slot = w * 2 + (unit_real_start <= start ? 0 : 1);
        if constexpr (!NARROW) {
            const float l_tot = halves_sum(st.l_run);
            const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
            constexpr int kPitch = D * 2 + 16;                   // LDS bytes per row (padded)
            constexpr int kRowChunks = D / 8;                     // 16-byte chunks per row
            constexpr int kRowsPerPass = kWave / kRowChunks;
            unsigned char *wbuf = g_ring + wave_u * kRowsPerWave * kPitch;
            #pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
                #pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    bf16x4 v;
                    #pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] = (__bf16)(st.o[dt][q4 * 4 + i] * inv);
                    *reinterpret_cast<bf16x4 *>(wbuf + col * kPitch + (dt * 32 + q4 * 8 + half * 4) * 2) = v;
                }
            #pragma unroll
            for (int k = 0; k < kRowsPerWave / kRowsPerPass; ++k) {
                const int r = k * kRowsPerPass + lane / kRowChunks, ch = lane % kRowChunks;
                const u32x4 v = *reinterpret_cast<const u32x4 *>(wbuf + r * kPitch + ch * 16);
                const int rl = wave_u * kRowsPerWave + r;           // row within the unit's block
                if (complete) {
                    const int ur = rb * p.rows_per_block + rl;
                    if (ur < rows_b) {
                        const int nd = ur / p.G, h = g * p.G + ur % p.G;
                        *reinterpret_cast<u32x4 *>(p.out + (((size_t)b * p.N + nd) * p.Hq + h) * D + ch * 8) = v;
                    }
                } else {
                    *reinterpret_cast<u32x4 *>(p.ws_o + ((size_t)slot * p.rows_per_block + rl) * D + ch * 8) = v;
                }
            }
            if (half == 0) {
                if (complete) {
                    if (row_ok && p.lse)
                        p.lse[((size_t)b * p.N + node) * p.Hq + hq] =
                            st.m_run * p.scale + __builtin_amdgcn_logf(l_tot) * kLn2;
                } else {
                    const int rloc = wave_u * kRowsPerWave + col;
                    float *pm = p.ws_ml + ((size_t)slot * p.rows_per_block + rloc) * 2;
                    pm[0] = (st.m_run == kNegInf) ? kNegInf : st.m_run * p.scale_log2;
                    pm[1] = l_tot;
                }
            }
        } else {
            // Narrow units: the waves' (max, sum, O^T) of the 16 rows meet in
            // the idle ring and combine with the log-sum-exp rule; thread
            // (row, 8-column chunk) writes one 16-byte piece of the row.
            constexpr int kCh = D / 8;
            float *ow = reinterpret_cast<float *>(g_ring);                 // [NW][16][D]
            float *mlw = ow + NW * 16 * D;                                  // [NW][16][2]
            const float lw = rows_sum(ns.l_run);
            #pragma unroll
            for (int db = 0; db < D / 16; ++db)
                *reinterpret_cast<f32x4 *>(ow + ((size_t)wave_u * 16 + (lane & 15)) * D + db * 16 +
                                           4 * (lane >> 4)) = ns.o[db];
            if (lane < 16) {
                mlw[(wave_u * 16 + lane) * 2] = ns.m_run;
                mlw[(wave_u * 16 + lane) * 2 + 1] = lw;
            }
            __syncthreads();
            const int nrows = min(16, rows_b);
            const float c = p.scale_log2;
            for (int task = tid; task < 16 * kCh; task += NT) {
                const int r = task / kCh, ch = task % kCh;
                if (r >= nrows) continue;
                float M = kNegInf;
                #pragma unroll
                for (int u = 0; u < NW; ++u) M = fmaxf(M, mlw[(u * 16 + r) * 2]);
                float Lsum = 0.f;
                float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
                #pragma unroll
                for (int u = 0; u < NW; ++u) {
                    const float mu = mlw[(u * 16 + r) * 2];
                    const float sc = (mu == kNegInf) ? 0.f : __builtin_amdgcn_exp2f((mu - M) * c);
                    Lsum += sc * mlw[(u * 16 + r) * 2 + 1];
                    const f32x4 a0 = *reinterpret_cast<const f32x4 *>(ow + ((size_t)u * 16 + r) * D + ch * 8);
                    const f32x4 a1 = *reinterpret_cast<const f32x4 *>(ow + ((size_t)u * 16 + r) * D + ch * 8 + 4);
                    #pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        acc[e] += sc * a0[e];
                        acc[4 + e] += sc * a1[e];
                    }
                }
                const float inv = Lsum > 0.f ? 1.f / Lsum : 0.f;
                bf16x8 o;
                #pragma unroll
                for (int e = 0; e < 8; ++e) o[e] = (__bf16)(acc[e] * inv);
                if (complete) {
                    const int nd = r / p.G, h = g * p.G + r % p.G;
                    *reinterpret_cast<bf16x8 *>(p.out + (((size_t)b * p.N + nd) * p.Hq + h) * D + ch * 8) = o;
                    if (ch == 0 && p.lse)
                        p.lse[((size_t)b * p.N + nd) * p.Hq + h] = M * p.scale + __builtin_amdgcn_logf(Lsum) * kLn2;
                } else {
                    *reinterpret_cast<bf16x8 *>(p.ws_o + ((size_t)slot * p.rows_per_block + r) * D + ch * 8) = o;
                    if (ch == 0) {
                        float *pm = p.ws_ml + ((size_t)slot * p.rows_per_block + r) * 2;
                        pm[0] = (M == kNegInf) ? kNegInf : M * c;
                        pm[1] = Lsum;
                    }
                }
            }
        }
        __syncthreads();                   // the ring is refilled by the next piece
    }

    // Rows of padding nodes (at or past a sequence's node count) are not part
    // of any unit: write them as zeros with lse -inf, a few nodes per workgroup.
    if (p.num_nodes) {
        const int chunks = p.Hq * D / 8;             // 16-byte chunks of one node's output
        for (int idx = w; idx < p.B * p.N; idx += p.num_wg) {
            const int b = idx / p.N, i = idx - b * p.N;
            if (i < g_nn[b]) continue;
            u16x8 *op = reinterpret_cast<u16x8 *>(p.out + ((size_t)b * p.N + i) * p.Hq * D);
            for (int c = tid; c < chunks; c += NT) op[c] = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
            if (p.lse)
                for (int h = tid; h < p.Hq; h += NT) p.lse[((size_t)b * p.N + i) * p.Hq + h] = kNegInf;
        }
    }
}

// Merge the pieces of every split unit. Block (chunk, h) serves the workgroup
// w that ran as block h of the main kernel, so it sits on the same XCD and
// finds the newest partials in that XCD's L2. If w finished a unit that began
// in an earlier share, the block merges a chunk of that unit's rows: one
// thread per (row, 8 head-dim lanes), pieces combined in workgroup order with
// an online log-sum-exp rescale (one pass, all loads of a piece independent).
template <int D>
__global__ __launch_bounds__(256) void tree_attention_merge_kernel(AttnParams p, int stride) {
    constexpr int D8 = D / 8;
    constexpr int kRowsPerWg = 256 / D8;
    const int h = blockIdx.x % stride;
    const int rchunk = blockIdx.x / stride;
    if (h >= p.num_wg) return;
    const int w = xcd_contiguous_id(h, p.num_wg);
    const i32x4 d = ((const CONST_AS i32x4 *)p.ws_desc)[w];
    const int b = d[0];
    if (b < 0) return;
    const int g = d[1], rb = d[2] & 0xFF, s0 = d[3];
    const int rows_b = (d[2] >> 8) * p.G;
    const int wf = s0 >> 1;

    const int rl = rchunk * kRowsPerWg + threadIdx.x / D8;
    const int d8 = threadIdx.x % D8;
    const int row = rb * p.rows_per_block + rl;
    if (rl >= p.rows_per_block || row >= rows_b) return;

    float M = kNegInf, den = 0.f;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    #pragma unroll 4
    for (int u = wf; u <= w; ++u) {
        // the first piece may sit in slot 1 of its workgroup; later ones start a share
        const int slot = u == wf ? s0 : u * 2;
        const size_t r = (size_t)slot * p.rows_per_block + rl;
        const f32x2 ml = *reinterpret_cast<const f32x2 *>(p.ws_ml + r * 2);
        const bf16x8 v = *reinterpret_cast<const bf16x8 *>(p.ws_o + r * D + d8 * 8);
        const float Mn = fmaxf(M, ml[0]);
        const float sc = (M == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(M - Mn);
        const float wt = (ml[0] == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(ml[0] - Mn) * ml[1];
        den = den * sc + wt;
        #pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = acc[i] * sc + wt * (float)v[i];
        M = Mn;
    }
    const int node = row / p.G;
    const int hq = g * p.G + row % p.G;
    const float inv = den > 0.f ? 1.f / den : 0.f;
    bf16x8 o;
    #pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = (__bf16)(acc[i] * inv);
    *reinterpret_cast<bf16x8 *>(p.out + (((size_t)b * p.N + node) * p.Hq + hq) * D + d8 * 8) = o;
    if (p.lse && d8 == 0)
        p.lse[((size_t)b * p.N + node) * p.Hq + hq] = (M + __builtin_amdgcn_logf(den)) * kLn2;
}

template <int D, int NW>
hipError_t launch_dn(const AttnParams &p, hipStream_t s) {
    hipError_t e;
    bool narrow_done = false;
    if constexpr (NW == 4) {
        if (p.narrow) {
            e = p.small_pages
                ? launch_kernel(tree_attention_kernel<D, NW, true, true>, dim3(p.num_wg), dim3(NW * kWave), s, p)
                : launch_kernel(tree_attention_kernel<D, NW, false, true>, dim3(p.num_wg), dim3(NW * kWave), s, p);
            narrow_done = true;
        }
    }
    if (!narrow_done)
        e = p.small_pages
            ? launch_kernel(tree_attention_kernel<D, NW, true, false>, dim3(p.num_wg), dim3(NW * kWave), s, p)
            : launch_kernel(tree_attention_kernel<D, NW, false, false>, dim3(p.num_wg), dim3(NW * kWave), s, p);
    if (e != hipSuccess) return e;
    if (p.num_wg > 1) {
        constexpr int kRowsPerWg = 256 / (D / 8);
        const int chunks = (p.rows_per_block + kRowsPerWg - 1) / kRowsPerWg;
        const int stride = (p.num_wg + kNumXcd - 1) / kNumXcd * kNumXcd;
        e = launch_kernel(tree_attention_merge_kernel<D>, dim3(stride * chunks), dim3(256), s, p,
                          stride);
    }
    return e;
}

template <int D>
hipError_t launch_d(const AttnParams &p, int waves, hipStream_t s) {
    switch (waves) {
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
