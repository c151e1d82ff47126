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
//     global_load_lds_dwordx4 (no register staging), two tiles ahead of the
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
//   * Tree visibility is a per-node ancestor bit set (256 bits) in LDS, built
//     by one wave with pointer doubling over the parent links while the first
//     tiles load; a masked score is replaced by -inf (selected, never added).
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
__device__ void build_ancestor_masks_wave(const AttnParams &p, int b) {
    const int lane = threadIdx.x & (kWave - 1);
    int j = -1;
    if (lane < p.N) {
        const int pi = p.parent[(size_t)b * p.N + lane];
        j = (pi < -1 || pi >= lane) ? -1 : pi;        // contract violation: treat as a root
    }
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
        }
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

    // Direct-to-LDS load of block i of this wave's share of one K (or V) tile
    // into ring stage `stage`.
    __device__ __forceinline__ void issue_one(const Blocks &bl, bool is_v, int stage, int wave_u,
                                              int i) const {
        unsigned char *dst = g_ring + stage * Gm::kStageBytes + (is_v ? Gm::kTileBytes : 0);
        const char *addr = (is_v ? bl.v[i] : bl.k[i]) + ((kib < bl.nv[i] ? row_off : 0u) + chunk_off[i]);
        __builtin_amdgcn_global_load_lds((const GLOBAL_AS void *)addr,
                                         (LDS_AS void *)(dst + (wave_u * LPT + i) * 1024), 16, 0, 0);
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

// Per-wave state of one segment: Q fragments (MFMA B operand), O^T
// accumulators, the current tile's scores and probabilities, running max/sum.
template <int D>
struct WaveState {
    static constexpr int NKS = D / 16;     // MFMA k-steps over the head dim
    static constexpr int NDT = D / 32;     // 32-wide head-dim tiles of the output
    bf16x8 qf[NKS];
    f32x16 o[NDT];
    f32x16 s[2];                           // S^T of the 2 x 32 keys of the tile
    bf16x8 pb[4];                          // P^T, 16 keys per k-step
    float m_run;                           // running max (raw score units)
    float l_run;                           // this lane's part of the running sum
};

// Matrix phase of one wave: O^T += V^T P^T for the previous tile (PV) and
// S^T = K Q^T for the current tile (SC). The ring reads are issued two
// groups ahead of the MFMAs that consume them; groups alternate PV / S so
// that consecutive MFMAs rarely depend on each other. hook(g) runs after
// group g: the caller issues its global->LDS tile loads there, a few at a
// time, instead of in one burst that would stall the wave.
template <int D, bool PV, bool SC, typename Hook>
__device__ __forceinline__ void matrix_phase(WaveState<D> &st, unsigned kaddr, unsigned vaddr,
                                             Hook &&hook) {
    using Gm = Geo<D>;
    constexpr int NKS = D / 16, NDT = D / 32, KH = NKS / 2;
    constexpr int C = Gm::kChunks;
    // group g: even g = PV k-step g/2, odd g = S quarter g/2 (half q/2, k-range q%2)
    constexpr int kGroups = 8;
    auto active = [](int gi) { return (gi & 1) ? SC : PV; };
    auto reads_of = [](int gi) { return (gi & 1) ? KH : 2 * NDT; };
    u32x2 vb[4][NDT][2];
    u32x4 kb[4][KH];
    auto issue = [&](int gi) {
        if (gi & 1) {
            const int q = gi >> 1, hf = q >> 1, part = q & 1;
            #pragma unroll
            for (int i = 0; i < KH; ++i) {
                const int ks = part * KH + i;
                asm volatile("ds_read_b128 %0, %1 offset:%2"
                             : "=v"(kb[q][i])
                             : "v"(kaddr ^ ((unsigned)ks << 5)), "i"(hf * 32 * Gm::kRowBytes));
            }
        } else {
            const int kk = gi >> 1;
            #pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
                #pragma unroll
                for (int rr = 0; rr < 2; ++rr) {
                    const unsigned flip = (unsigned)((dt * 4) ^ swz<C>((rr * 8) % C)) << 4;
                    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2"
                                 : "=v"(vb[kk][dt][rr])
                                 : "v"(vaddr ^ flip), "i"((kk * 16 + rr * 8) * Gm::kRowBytes));
                }
        }
    };
    auto consume = [&](int gi) {
        if (gi & 1) {
            const int q = gi >> 1, hf = q >> 1, part = q & 1;
            #pragma unroll
            for (int i = 0; i < KH; ++i) {
                tie(kb[q][i]);
                st.s[hf] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, kb[q][i]), st.qf[part * KH + i], st.s[hf], 0, 0, 0);
            }
        } else {
            const int kk = gi >> 1;
            #pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                tie(vb[kk][dt][0]);
                tie(vb[kk][dt][1]);
                const u32x4 a = {vb[kk][dt][0][0], vb[kk][dt][0][1], vb[kk][dt][1][0], vb[kk][dt][1][1]};
                st.o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, a), st.pb[kk], st.o[dt], 0, 0, 0);
            }
        }
    };
    if (SC) {
        #pragma unroll
        for (int hf = 0; hf < 2; ++hf)
            #pragma unroll
            for (int r = 0; r < 16; ++r) st.s[hf][r] = 0.f;
    }
    // active groups in order; next(gi) = following active group (or kGroups)
    auto next = [&](int gi) {
        int n = gi + 1;
        while (n < kGroups && !active(n)) ++n;
        return n;
    };
    const int g0 = next(-1);
    const int g1 = next(g0);
    issue(g0);
    if (g1 < kGroups) issue(g1);
    #pragma unroll
    for (int gi = 0; gi < kGroups; ++gi) {
        if (active(gi)) {
            const int gn = next(gi);
            lds_wait_n(gn < kGroups ? reads_of(gn) : 0);
            consume(gi);
            const int gnn = gn < kGroups ? next(gn) : kGroups;
            if (gnn < kGroups) issue(gnn);
        }
        hook(gi);          // the caller's tile loads, spread over the phase
    }
}

// Softmax phase of one wave for tile t: mask, tile max, lazy rescale of the
// running state, exponentials into P^T (bf16) and the running sum.
template <int D>
__device__ __forceinline__ void softmax_phase(WaveState<D> &st, const AttnParams &p, int t,
                                              int ntp, int L, int node, int half) {
    constexpr int NDT = D / 32;
    // Lane holds keys hf*32 + (r/4)*8 + half*4 + r%4 of its row.
    if (t < ntp) {
        const int lim_t = L - t * KT;                   // keys >= lim_t are past the prefix
        if (lim_t < KT) {                               // wave-uniform: only the last prefix tile
            const int lim = lim_t - half * 4;
            #pragma unroll
            for (int hf = 0; hf < 2; ++hf)
                #pragma unroll
                for (int r = 0; r < 16; ++r)
                    st.s[hf][r] = (hf * 32 + (r >> 2) * 8 + (r & 3) >= lim) ? kNegInf : st.s[hf][r];
        }
    } else {
        const unsigned long long vis = g_anc[node][t - ntp] >> (half * 4);
        #pragma unroll
        for (int hf = 0; hf < 2; ++hf)
            #pragma unroll
            for (int r = 0; r < 16; ++r)
                st.s[hf][r] = ((vis >> (hf * 32 + (r >> 2) * 8 + (r & 3))) & 1ull) ? st.s[hf][r] : kNegInf;
    }
    // The running max is only raised when a score exceeds it by more than
    // kRescaleSlack (log2 units), so O is rarely rescaled. The tile max is a
    // tree of three-input maxes.
    float v[32];
    #pragma unroll
    for (int r = 0; r < 16; ++r) {
        v[r] = st.s[0][r];
        v[16 + r] = st.s[1][r];
    }
    float m1[12];
    #pragma unroll
    for (int i = 0; i < 10; ++i) m1[i] = max3(v[3 * i], v[3 * i + 1], v[3 * i + 2]);
    m1[10] = v[30];
    m1[11] = v[31];
    const float m2a = max3(m1[0], m1[1], m1[2]), m2b = max3(m1[3], m1[4], m1[5]);
    const float m2c = max3(m1[6], m1[7], m1[8]), m2d = max3(m1[9], m1[10], m1[11]);
    const float tmax = halves_max(max3(m2a, m2b, fmaxf(m2c, m2d)));
    const bool raise = tmax * p.scale_log2 > st.m_run * p.scale_log2 + kRescaleSlack;
    if (__any(raise)) {
        const float m_new = raise ? tmax : st.m_run;
        const float alpha = (st.m_run == kNegInf) ? 0.f
                            : __builtin_amdgcn_exp2f((st.m_run - m_new) * p.scale_log2);
        st.l_run *= alpha;
        #pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
            #pragma unroll
            for (int r = 0; r < 16; ++r) st.o[dt][r] *= alpha;
        st.m_run = m_new;
    }
    const float msc = (st.m_run == kNegInf) ? 0.f : st.m_run * p.scale_log2;
    float ps[4] = {0.f, 0.f, 0.f, 0.f};
    #pragma unroll
    for (int kk = 0; kk < 4; ++kk)
        #pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float x = __builtin_amdgcn_exp2f(
                __builtin_fmaf(st.s[kk >> 1][(kk & 1) * 8 + e], p.scale_log2, -msc));
            ps[e & 3] += x;
            st.pb[kk][e] = (__bf16)x;
        }
    st.l_run += (ps[0] + ps[1]) + (ps[2] + ps[3]);
}

// Barrier between the phases of the two wave groups; nothing is scheduled
// across it.
__device__ __forceinline__ void phase_barrier() {
    __builtin_amdgcn_sched_barrier(0);
    lds_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

template <int D, int NW, bool SMALL>
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
    // Two wave groups run half a tile apart: while one group is in its matrix
    // phase the other is in its softmax phase, so every SIMD has MFMA and VALU
    // work from different waves at the same time.
    const int grp = (NW >= 2 && wave_u >= NW / 2) ? 1 : 0;
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
        const int t0 = max(off - C, 0);
        const int t_end = v_end - C;
        if (t_end <= t0) continue;                    // only set-up tiles of this unit
        const bool complete = (t0 == 0 && t_end == ulen);

        // ---- this wave's 32 query rows: Q fragments stay in registers
        const int row = rb * p.rows_per_block + wave_u * kRowsPerWave + col;
        const bool row_ok = row < rows_b;
        const int node = row_ok ? row / p.G : 0;
        const int hq = g * p.G + (row_ok ? row % p.G : 0);
        WaveState<D> st;
        {
            const uint16_t *qp = p.q + (((size_t)b * p.N + node) * p.Hq + hq) * D + half * 8;
            #pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
                u16x8 v = row_ok ? *reinterpret_cast<const u16x8 *>(qp + ks * 16)
                                 : u16x8{0, 0, 0, 0, 0, 0, 0, 0};
                st.qf[ks] = __builtin_bit_cast(bf16x8, v);
            }
        }
        #pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
            #pragma unroll
            for (int r = 0; r < 16; ++r) st.o[dt][r] = 0.f;
        st.m_run = kNegInf;
        st.l_run = 0.f;

        const int npages = (L + p.P - 1) >> p.p_shift;
        const bool has_tree = t_end > ntp;
        auto kaddr_of = [&](int t) { return ring_base + (t & (NS - 1)) * Gm::kStageBytes + k_lane; };
        auto vaddr_of = [&](int t) {
            return ring_base + (t & (NS - 1)) * Gm::kStageBytes + Gm::kTileBytes + v_lane;
        };

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
            const bool want_anc = first && has_tree && anc_b != b;
            if (SMALL && ta < ntp) load_pages<NT>(p, b, page_first, npages);

            const int T = tb - ta;
            // Load batch i = K tile ta+i and V tile ta+i-1 (those that exist). It is
            // issued two tile periods before the matrix phase that first needs it
            // (a third period ahead measured 2 % slower: the extra loads in flight
            // only lengthen the issue stalls).
            auto batch_loads = [&](int i) {
                return ((i >= 0 && i < T) ? LPT : 0) + ((i >= 1 && i <= T) ? LPT : 0);
            };
            // pk: page ids of the K tile of the next batch (fetched one tile
            // period ahead); last: blocks of the last issued K tile, which is
            // the V tile of the next batch.
            int pk[LPT];
            typename Issue::Blocks last;
            auto issue_batch = [&](int i) {
                const int tk = ta + i, tv = ta + i - 1;
                if (SMALL) {
                    if (i < T) {
                        if (tk < ntp) ld.issue_small(p, tk, false, page_first, wave_u);
                        else ld.issue(ld.blocks(p, tk, wave_u, pk), false, tk & (NS - 1), wave_u);
                    }
                    if (i >= 1 && i <= T) {
                        if (tv < ntp) ld.issue_small(p, tv, true, page_first, wave_u);
                        else ld.issue(ld.blocks(p, tv, wave_u, pk), true, tv & (NS - 1), wave_u);
                    }
                    return;
                }
                typename Issue::Blocks cur;
                if (i < T) {
                    cur = ld.blocks(p, tk, wave_u, pk);
                    ld.issue(cur, false, tk & (NS - 1), wave_u);
                }
                if (i >= 1 && i <= T) ld.issue(last, true, tv & (NS - 1), wave_u);
                last = cur;
            };
            auto fetch = [&](int i) { ld.fetch_pages(p, b, ta + i, wave_u, pk); };

            // Q (issued above) and the first tiles are in flight together: the
            // first tile wait below also covers Q, which was issued earlier.
            ld.set_unit(p, b, g, L, ntp, nodes);
            {
                int ids[3][LPT];
                #pragma unroll
                for (int i = 0; i < 3; ++i) ld.fetch_pages(p, b, ta + i, wave_u, ids[i]);
                #pragma unroll
                for (int i = 0; i < 3; ++i) {
                    #pragma unroll
                    for (int k = 0; k < LPT; ++k) pk[k] = ids[i][k];
                    if (i < 2) issue_batch(i);    // pk then holds the ids of batch 2
                }
            }
            // Ancestor sets, while the loads above are in flight, by one wave
            // (the other waves only read them at the tree tiles, after several
            // workgroup barriers): in registers up to 64 nodes, else in LDS.
            if (want_anc) {
                if (wave_u == 0) {
                    if (p.N <= kWave) build_ancestor_masks_wave(p, b);
                    else build_ancestor_masks_wave_lds(p, b);
                }
                anc_b = b;
            }

            // Slots of half a tile period, separated by workgroup barriers. Group 0
            // runs matrix j in slot 2j and softmax j in slot 2j+1; group 1 runs
            // the same instruction stream one slot later (one extra barrier at
            // its start, one at group 0's end). Batch j must have landed, for
            // every wave, before slot 2j: group 0 waits before the barrier that
            // opens its matrix j, group 1 before the one that opens its softmax
            // j-1. Both groups issue batch j+2 when they start matrix j; the
            // ring stages it overwrites were last read in slot 2j-3.
            if (grp == 1) {
                wait_vm_at_most(batch_loads(1));
                phase_barrier();
            }
            // slot pair j: barrier, matrix j (issuing batch j+2 along the way);
            // barrier, softmax j
            typename Issue::Blocks cur;
            bool have_k = false, have_v = false;
            int stage_k = 0, stage_v = 0;
            // Waits: batch j (group 0, before matrix j) or batch j+1 (group 1,
            // before softmax j) complete, leaving this wave's loads of the one
            // later batch in flight.
            auto open_matrix = [&](int j) {
                if (grp == 0) wait_vm_at_most(batch_loads(j + 1));
                phase_barrier();
                // The matrix phase runs at raised wave priority: when both waves of
                // a SIMD could issue, its MFMAs and LDS reads go first and the other
                // group's softmax fills the gaps.
                __builtin_amdgcn_s_setprio(1);
                const int i = j + 2;
                have_k = have_v = false;
                if (i <= T) {
                    if (SMALL) {
                        issue_batch(i);
                    } else {
                        have_k = i < T;
                        have_v = true;
                        stage_k = (ta + i) & (NS - 1);
                        stage_v = (ta + i - 1) & (NS - 1);
                        if (have_k) cur = ld.blocks(p, ta + i, wave_u, pk);
                    }
                }
            };
            // Loads of batch j+2 during matrix j: full batches in the steady
            // state, the tail checks which halves exist.
            auto hook_full = [&](int gi) {
                if (SMALL) return;
                #pragma unroll
                for (int k = 0; k < 2 * LPT; ++k) {
                    if (k * 8 / (2 * LPT) != gi) continue;
                    if (k < LPT) ld.issue_one(cur, false, stage_k, wave_u, k);
                    else ld.issue_one(last, true, stage_v, wave_u, k - LPT);
                }
            };
            auto hook = [&](int gi) {
                if (SMALL) return;
                #pragma unroll
                for (int k = 0; k < 2 * LPT; ++k) {
                    if (k * 8 / (2 * LPT) != gi) continue;
                    if (k < LPT) {
                        if (have_k) ld.issue_one(cur, false, stage_k, wave_u, k);
                    } else if (have_v) {
                        ld.issue_one(last, true, stage_v, wave_u, k - LPT);
                    }
                }
            };
            auto close_matrix = [&]() {
                if (!SMALL && have_v) last = cur;
            };
            auto softmax = [&](int j) {
                if (grp == 1) wait_vm_at_most(batch_loads(j + 2));
                __builtin_amdgcn_s_setprio(0);
                phase_barrier();
                softmax_phase<D>(st, p, ta + j, ntp, L, node, half);
                fetch(j + 3);          // ids for the batch issued at the next matrix phase
            };
            open_matrix(0);
            matrix_phase<D, false, true>(st, kaddr_of(ta), 0u, hook);
            close_matrix();
            softmax(0);
            int j = 1;
            for (; j + 2 < T; ++j) {                 // batch j+2 is full
                open_matrix(j);
                matrix_phase<D, true, true>(st, kaddr_of(ta + j), vaddr_of(ta + j - 1), hook_full);
                close_matrix();
                softmax(j);
            }
            for (; j < T; ++j) {
                open_matrix(j);
                matrix_phase<D, true, true>(st, kaddr_of(ta + j), vaddr_of(ta + j - 1), hook);
                close_matrix();
                softmax(j);
            }
            open_matrix(T);
            matrix_phase<D, true, false>(st, 0u, vaddr_of(ta + T - 1), hook);
            if (grp == 0 && NW >= 2) phase_barrier();
            ta = tb;
            __syncthreads();               // ring and page ids are reused next
        }

        // ---- finish the segment
        const float l_tot = halves_sum(st.l_run);
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
                        for (int i = 0; i < 4; ++i) v[i] = (__bf16)(st.o[dt][q4 * 4 + i] * inv);
                        *reinterpret_cast<bf16x4 *>(op + dt * 32 + q4 * 8 + half * 4) = v;
                    }
                if (p.lse && half == 0)
                    p.lse[((size_t)b * p.N + node) * p.Hq + hq] =
                        st.m_run * p.scale + __builtin_amdgcn_logf(l_tot) * kLn2;
            }
        } else {
            // A piece of a split unit: its output normalised by its own sum, in
            // bf16, plus the (max, sum) pair in fp32. Slot 0 holds the piece that
            // continues a unit from before this share, slot 1 the one that starts
            // inside it.
            const int slot = w * 2 + (unit_real_start <= start ? 0 : 1);
            const int rloc = wave_u * kRowsPerWave + col;
            uint16_t *po = p.ws_o + ((size_t)slot * p.rows_per_block + rloc) * D;
            const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
            #pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
                #pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    bf16x4 v;
                    #pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] = (__bf16)(st.o[dt][q4 * 4 + i] * inv);
                    *reinterpret_cast<bf16x4 *>(po + dt * 32 + q4 * 8 + half * 4) = v;
                }
            if (half == 0) {
                float *pm = p.ws_ml + ((size_t)slot * p.rows_per_block + rloc) * 2;
                pm[0] = (st.m_run == kNegInf) ? kNegInf : st.m_run * p.scale_log2;
                pm[1] = l_tot;
            }
        }
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
    hipError_t e = p.small_pages
        ? launch_kernel(tree_attention_kernel<D, NW, true>, dim3(p.num_wg), dim3(NW * kWave), s, p)
        : launch_kernel(tree_attention_kernel<D, NW, false>, dim3(p.num_wg), dim3(NW * kWave), s, p);
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
