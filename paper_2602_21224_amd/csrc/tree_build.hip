// Draft-tree builder for gfx950: token-info sampling (Alg. 1) followed by the
// verification-budget pruning (§5.2). It produces the parent / token arrays
// (and per-sequence node counts) that the verification calls consume.
//
// At step i a frontier node's children are the k most probable tokens of
// softmax(l_i + r), r being the node token's row of the hot-token table (§5.1
// collapses the token-info embedding into an additive logit table; §6.1 keeps
// it for the hot tokens only). Everything about that softmax that does not
// depend on the node -- the non-hot entries of l_i -- is reduced once per
// (sequence, step), for all steps at once (tb_rows_kernel, one streaming pass
// over the logits). Per step only the H hot columns are visited for each
// frontier node (tb_expand_kernel), and one workgroup per sequence combines
// the partial results into children, joint probabilities and the next
// frontier (tb_select_kernel). tb_prune_kernel finally keeps the `budget`
// nodes of largest joint probability, in creation order.
//
// Decisions: candidates are ranked by the fp32 sum l + r (the precision of the
// logits; ties to the lower vocabulary id) through a packed 64-bit key.
// Probabilities and joint probabilities are fp64 (exp and sums in double), so
// frontier and pruning decisions agree with an fp64 evaluation unless two
// joint probabilities are equal to within about 1e-13.
#include "tv_internal.h"

namespace tv {
namespace {

constexpr int kTbThreads = 256;
constexpr int kTbChunk = 32;               // candidates per thread held in registers at once
constexpr int kExpThreads = kWave;         // one wave per expansion workgroup: no block reduction
constexpr int kTbWaves = kTbThreads / kWave;
constexpr int kPruneThreads = 1024;
constexpr int kPruneSlots = 4096;          // >= 1 + k + (S - 1) k^2 for k, S <= 16

// One partial reduction over a set of candidates: their maximum, the sum of
// exp(x - max) in fp64, and the top-k keys in descending order (0 = none).
struct TbPart {
    float m;
    int pad;
    double s;
    unsigned long long key[kTbMaxK];
};

// The frontier of one sequence: its node count and, per slot (frontier order),
// the node, its token, the token's hot row (-1: none) and its joint
// probability -- everything the next expansion and selection need, in one
// load (no chain through the node arrays and the hot map).
struct TbSlot {
    int node, tok, h, pad;
    double joint;
};
struct TbFrontier {
    int count, pad[3];
    TbSlot slot[kTbMaxK];
};

// Hot row of token t (-1 when it has none).
__device__ __forceinline__ int hot_row(const int32_t *hot_index, int t, int V, int H) {
    int h = (H > 0 && t >= 0 && t < V) ? hot_index[t] : -1;
    return h >= H ? -1 : h;
}

__device__ __forceinline__ unsigned long long umax64(unsigned long long a, unsigned long long b) {
    return a > b ? a : b;
}

__device__ __forceinline__ float key_value(unsigned long long key) {
    const unsigned int k = (unsigned int)(key >> 32);
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

__device__ __forceinline__ int key_index(unsigned long long key) {
    return (int)(0xFFFFFFFFu - (unsigned int)key);
}

__device__ __forceinline__ double exp_nonpos(double x, const double *tab);

// Running (max, sum of exp(x - max)) of one thread, fp64 sums; a batch of
// values is folded in with one rescale, without per-value branches. tab: the
// 2^(j/32) table of exp_nonpos.
struct OnlineSum {
    float m = -__builtin_huge_valf();
    double s = 0.0;
    __device__ __forceinline__ void merge(float m2, double s2, const double *tab) {
        if (m2 == -__builtin_huge_valf()) return;
        if (m == -__builtin_huge_valf()) { m = m2; s = s2; return; }
        const float mn = fmaxf(m, m2);
        s = s * exp_nonpos((double)m - (double)mn, tab) + s2 * exp_nonpos((double)m2 - (double)mn, tab);
        m = mn;
    }
};

// Cross-lane helpers without LDS: readlane (wave-uniform source lane) and a
// one-lane shift inside each row of 16 lanes (DPP row_shr:1).
__device__ __forceinline__ unsigned long long readlane64(unsigned long long v, int src) {
    const unsigned int lo = __builtin_amdgcn_readlane((int)(unsigned int)v, src);
    const unsigned int hi = __builtin_amdgcn_readlane((int)(unsigned int)(v >> 32), src);
    return ((unsigned long long)hi << 32) | lo;
}

__device__ __forceinline__ unsigned long long row_shr1_64(unsigned long long v) {
    const int lo = (int)(unsigned int)v, hi = (int)(unsigned int)(v >> 32);
    const unsigned int nlo = __builtin_amdgcn_update_dpp(lo, lo, 0x111, 0xF, 0xF, false);
    const unsigned int nhi = __builtin_amdgcn_update_dpp(hi, hi, 0x111, 0xF, 0xF, false);
    return ((unsigned long long)nhi << 32) | nlo;
}

// Largest 64-bit key over the wave, by a scan of per-row maxima (no LDS).
__device__ __forceinline__ unsigned long long wave_max64(unsigned long long v) {
    #pragma unroll
    for (int sh = 1; sh < 16; sh <<= 1) {        // row_shr:sh; lanes below sh keep their value
        const int lo = (int)(unsigned int)v, hi = (int)(unsigned int)(v >> 32);
        const unsigned int nlo = sh == 1 ? __builtin_amdgcn_update_dpp(lo, lo, 0x111, 0xF, 0xF, false)
                               : sh == 2 ? __builtin_amdgcn_update_dpp(lo, lo, 0x112, 0xF, 0xF, false)
                               : sh == 4 ? __builtin_amdgcn_update_dpp(lo, lo, 0x114, 0xF, 0xF, false)
                                         : __builtin_amdgcn_update_dpp(lo, lo, 0x118, 0xF, 0xF, false);
        const unsigned int nhi = sh == 1 ? __builtin_amdgcn_update_dpp(hi, hi, 0x111, 0xF, 0xF, false)
                               : sh == 2 ? __builtin_amdgcn_update_dpp(hi, hi, 0x112, 0xF, 0xF, false)
                               : sh == 4 ? __builtin_amdgcn_update_dpp(hi, hi, 0x114, 0xF, 0xF, false)
                                         : __builtin_amdgcn_update_dpp(hi, hi, 0x118, 0xF, 0xF, false);
        v = umax64(v, ((unsigned long long)nhi << 32) | nlo);
    }
    // lane 15 of every row now holds its row's maximum
    return umax64(umax64(readlane64(v, 15), readlane64(v, 31)),
                  umax64(readlane64(v, 47), readlane64(v, 63)));
}

// Largest 32-bit value over the wave: a scan of per-row maxima by DPP row
// shifts, then the four rows' last lanes (no LDS).
__device__ __forceinline__ unsigned int wave_max32(unsigned int v) {
    v = max(v, (unsigned int)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x111, 0xF, 0xF, false));
    v = max(v, (unsigned int)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x112, 0xF, 0xF, false));
    v = max(v, (unsigned int)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x114, 0xF, 0xF, false));
    v = max(v, (unsigned int)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x118, 0xF, 0xF, false));
    // lane 15 of every row now holds its row's maximum
    return max(max((unsigned int)__builtin_amdgcn_readlane((int)v, 15), (unsigned int)__builtin_amdgcn_readlane((int)v, 31)),
               max((unsigned int)__builtin_amdgcn_readlane((int)v, 47), (unsigned int)__builtin_amdgcn_readlane((int)v, 63)));
}

// Whole-wave reductions without LDS: butterflies inside each row of 16 lanes
// by DPP (swap neighbours, swap pairs, mirror each half row, mirror the row:
// after each step every lane of the group holds the group's result), then
// across rows by the row-pair and half-wave swaps. Every lane ends with the
// result.
template <int C>
__device__ __forceinline__ unsigned int dpp32(unsigned int v) {
    return (unsigned int)__builtin_amdgcn_update_dpp((int)v, (int)v, C, 0xF, 0xF, false);
}
template <int C>
__device__ __forceinline__ double dpp64(double v) {
    const unsigned long long b = (unsigned long long)__double_as_longlong(v);
    const unsigned int lo = dpp32<C>((unsigned int)b), hi = dpp32<C>((unsigned int)(b >> 32));
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

__device__ __forceinline__ float wave_allmax(float v) {
    v = fmaxf(v, __uint_as_float(dpp32<kDppXor1>(__float_as_uint(v))));
    v = fmaxf(v, __uint_as_float(dpp32<kDppXor2>(__float_as_uint(v))));
    v = fmaxf(v, __uint_as_float(dpp32<kDppHalfMirror>(__float_as_uint(v))));
    v = fmaxf(v, __uint_as_float(dpp32<kDppMirror>(__float_as_uint(v))));
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    const auto h = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(h[0]), __uint_as_float(h[1]));
}

__device__ __forceinline__ double wave_allsum(double v) {
    v += dpp64<kDppXor1>(v);
    v += dpp64<kDppXor2>(v);
    v += dpp64<kDppHalfMirror>(v);
    v += dpp64<kDppMirror>(v);
    #pragma unroll
    for (int half = 0; half < 2; ++half) {         // row pairs, then the wave's halves
        const unsigned long long b = (unsigned long long)__double_as_longlong(v);
        const unsigned int lo = (unsigned int)b, hi = (unsigned int)(b >> 32);
        const auto l = half == 0 ? __builtin_amdgcn_permlane16_swap(lo, lo, false, false)
                                 : __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
        const auto h = half == 0 ? __builtin_amdgcn_permlane16_swap(hi, hi, false, false)
                                 : __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
        v = __longlong_as_double((long long)(((unsigned long long)h[0] << 32) | l[0])) +
            __longlong_as_double((long long)(((unsigned long long)h[1] << 32) | l[1]));
    }
    return v;
}

// Sum over aligned groups of n consecutive lanes (n = 1, 2, 4, 8 or 16,
// wave-uniform); every lane of a group ends with the group's sum.
__device__ __forceinline__ int group_sum(int v, int n) {
    if (n >= 2) v += (int)dpp32<kDppXor1>((unsigned int)v);
    if (n >= 4) v += (int)dpp32<kDppXor2>((unsigned int)v);
    if (n >= 8) v += (int)dpp32<kDppHalfMirror>((unsigned int)v);
    if (n >= 16) v += (int)dpp32<kDppMirror>((unsigned int)v);
    return v;
}

// A wave's top-k list, distributed over lanes: lane j < k holds the (j+1)-th
// largest key seen by the wave (0 = empty). The k-th key is the wave's
// admission threshold, so after the first few batches almost no candidate
// needs more than one compare; an admitted key is inserted by one shift.
struct WaveTopK {
    unsigned long long w = 0ull;      // this lane's entry
    unsigned long long thr = 0ull;    // the k-th entry (wave-uniform)
    __device__ __forceinline__ void offer(unsigned long long cand, int k, int lane) {
        unsigned long long mask = __ballot(cand > thr);
        while (mask) {                                   // wave-uniform
            const int src = __builtin_ctzll(mask);
            const unsigned long long cc = readlane64(cand, src);
            const int pos = __popcll(__ballot(lane < k && w > cc));   // entries above cc
            const unsigned long long up = row_shr1_64(w);
            if (lane < k) w = lane == pos ? cc : (lane > pos ? up : w);
            thr = readlane64(w, k - 1);
            mask &= ~(1ull << src);
            mask &= __ballot(cand > thr);
        }
    }
};

// exp(x) for x <= 0 in double precision, by Tang's table-driven method (ACM
// TOMS 15(2), 1989): x = (32 n + j) ln2/32 + r with |r| <= ln2/64, so
// e^x = 2^(n >> 5) 2^(j/32) e^r, j = n & 31; e^r - 1 from its degree-6 Taylor
// polynomial (truncation below 2e-17 on that interval); 2^(j/32) from a
// 32-entry table (tab, filled by fill_exp2_table). ln2/32 is split into
// kL1 (its 37 leading significant bits, so N kL1 is exact for |N| < 2^16) and
// kL2 = ln2/32 - kL1 rounded to double. Arguments below -745 (and -inf) give 0.
// About 1 ulp, against about 45 instructions for the library's exp.
__device__ __forceinline__ double exp_nonpos(double x, const double *tab) {
    const double kInvL = 46.16624130844683;          // 32 / ln2
    const double kL1 = 0.021660849392446835;
    const double kL2 = 5.145609244655338e-14;
    const double N = __builtin_rint(x * kInvL);
    double r = __builtin_fma(-N, kL1, x);
    r = __builtin_fma(-N, kL2, r);
    double q = __builtin_fma(r, 1.0 / 720.0, 1.0 / 120.0);
    q = __builtin_fma(q, r, 1.0 / 24.0);
    q = __builtin_fma(q, r, 1.0 / 6.0);
    q = __builtin_fma(q, r, 0.5);
    q = __builtin_fma(q, r, 1.0);
    q *= r;                                          // e^r - 1
    const int n = x < -745.0 ? 0 : (int)N;
    const double t = tab[n & 31];
    const double y = __builtin_ldexp(__builtin_fma(t, q, t), n >> 5);
    return x < -745.0 ? 0.0 : y;
}

// 2^(j/32), j = 0..31, into LDS for exp_nonpos; the caller synchronises.
__device__ __forceinline__ void fill_exp2_table(double *tab) {
    if (threadIdx.x < 32) tab[threadIdx.x] = exp2((double)threadIdx.x / 32.0);
}

// One chunk of a thread's candidates, all in registers: x[u] is the value of
// vocabulary id id(u), -inf when it is not a candidate. Folds their
// (max, fp64 sum of exp(x - max)) into os and their k largest keys into the
// wave's list. The wave's k largest are all at or above the k-th largest of
// the lanes' maxima (those are k candidates already), so only candidates at or
// above that floor form keys and go through the wave-serial insertion.
template <int U, typename Id>
__device__ __forceinline__ void fold_chunk(const float (&x)[U], Id id, int k, int lane,
                                           const double *tab, OnlineSum &os, WaveTopK &tk) {
    constexpr float kNegInf = -__builtin_huge_valf();
    float m = kNegInf;
    unsigned int kv[U];
    unsigned int kmax = 0u;
    #pragma unroll
    for (int u = 0; u < U; ++u) {
        m = fmaxf(m, x[u]);
        kv[u] = x[u] != kNegInf ? order_key(x[u]) : 0u;
        kmax = max(kmax, kv[u]);
    }
    if (m != kNegInf) {
        double sum = 0.0;
        #pragma unroll
        for (int u = 0; u < U; ++u) sum += exp_nonpos((double)x[u] - (double)m, tab);
        os.merge(m, sum, tab);
    }
    // k-th largest lane maximum (ties may remove two lanes in one round: the
    // floor only gets lower, never wrong); once the wave's list is full, its
    // k-th key is a floor already and the rounds are skipped
    unsigned int floor_key = (unsigned int)(tk.thr >> 32);
    if (floor_key == 0u) {
        for (int r = 0; r < k; ++r) {
            const unsigned int mx = wave_max32(kmax);
            if (kmax == mx) kmax = 0u;
            floor_key = mx;
        }
    }
    #pragma unroll
    for (int u = 0; u < U; ++u) {
        const bool pass = kv[u] != 0u && kv[u] >= floor_key;
        if (__ballot(pass) == 0ull) continue;                 // wave-uniform
        tk.offer(pass ? pack_key(kv[u], (unsigned int)id(u)) : 0ull, k, lane);
    }
}

// Workgroup reduction of every thread's OnlineSum and every wave's top-k list
// into one TbPart.
__device__ void block_reduce_part(OnlineSum os, const WaveTopK &tk, int k, TbPart *out,
                                  const double *tab) {
    __shared__ float s_m[kTbWaves];
    __shared__ double s_s[kTbWaves];
    __shared__ unsigned long long s_key[kTbWaves * kTbMaxK];
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    // the wave's maximum first, then each lane's sum rescaled to it once and
    // the sums added (one exponential per lane instead of one per merge)
    const float wm = wave_allmax(os.m);
    const double ws = wave_allsum(os.m == -__builtin_huge_valf() ? 0.0 : os.s * exp_nonpos((double)os.m - (double)wm, tab));
    os.m = wm;
    os.s = ws;
    if (lane == 0) { s_m[wave] = os.m; s_s[wave] = os.s; }
    if (lane < kTbMaxK) s_key[wave * kTbMaxK + lane] = lane < k ? tk.w : 0ull;
    __syncthreads();
    if (wave == 0) {
        // the k largest of the waves' lists: one candidate per lane
        unsigned long long c = lane < kTbWaves * kTbMaxK ? s_key[lane] : 0ull;
        for (int r = 0; r < k; ++r) {
            const unsigned long long best = wave_max64(c);
            if (c == best) c = 0ull;
            if (lane == 0) out->key[r] = best;
        }
        if (lane == 0) {
            for (int r = k; r < kTbMaxK; ++r) out->key[r] = 0ull;
            OnlineSum t;
            for (int w = 0; w < kTbWaves; ++w) t.merge(s_m[w], s_s[w], tab);
            out->m = t.m;
            out->pad = 0;
            out->s = t.s;
        }
    }
}

// One wave's OnlineSum and top-k list into one TbPart (the wave maximum first,
// then each lane's sum rescaled to it once; the list is already in lanes
// 0..k-1).
__device__ __forceinline__ void wave_reduce_part(const OnlineSum &os, const WaveTopK &tk, int k,
                                                 int lane, TbPart *out, const double *tab) {
    const float wm = wave_allmax(os.m);
    const double ws = wave_allsum(os.m == -__builtin_huge_valf() ? 0.0 : os.s * exp_nonpos((double)os.m - (double)wm, tab));
    if (lane == 0) { out->m = wm; out->pad = 0; out->s = ws; }
    if (lane < kTbMaxK) out->key[lane] = lane < k ? tk.w : 0ull;
}

// Steps of sequence b: logits rows [first, first + count). A first tree uses all
// S rows. A re-sampled tree (Alg. 2; accept_len given) starts after the first
// rejected position -- the accepted path counts the root, so that position is
// accept_len and the remaining rows are accept_len .. S-1 -- and is the single
// ground-truth node unless more than r rows remain. A sequence that verified
// nothing has no tree (count -1).
struct TbWindow {
    int first, count;
};

__device__ __forceinline__ TbWindow tb_window(const int32_t *accept_len, int b, int S, int r) {
    if (!accept_len) return {0, S};
    const int a = accept_len[b];
    if (a <= 0) return {0, -1};
    const int remain = S - a;
    return {min(a, S), remain > r ? remain : 0};
}

// Node-independent part of every (sequence, step): the non-hot tokens of the
// step's logits, one segment of the vocabulary per workgroup. Workgroup
// (row (b, 0), segment 0) also places the root and the first frontier.
__global__ __launch_bounds__(kTbThreads) void tb_rows_kernel(
    const float *__restrict__ logits, const int32_t *__restrict__ hot_vocab,
    const int32_t *__restrict__ hot_index, const int32_t *__restrict__ root_token,
    const int32_t *__restrict__ accept_len, int r, int S, int V, int H, int k, int seg_len,
    TbPart *__restrict__ rows, float *__restrict__ hot_logits, int max_nodes,
    int32_t *__restrict__ node_tok, int32_t *__restrict__ node_par,
    double *__restrict__ node_joint, TbFrontier *__restrict__ frontier) {
    __shared__ double s_exp2[32];
    fill_exp2_table(s_exp2);
    __syncthreads();
    const int row = blockIdx.x, seg = blockIdx.y;
    const int v0 = seg * seg_len, v1 = min(V, v0 + seg_len);
    const float *l = logits + (size_t)row * V;
    OnlineSum os;
    WaveTopK tk;
    const int lane = threadIdx.x & (kWave - 1);
    // Chunks of kTbChunk tokens per thread, every load of a chunk issued before
    // any is used (indices clamped, so the loads are unconditional). The chunk
    // loop is uniform over the workgroup (the wave's list is updated by
    // whole-wave steps).
    const int iters = (max(v1 - v0, 0) + kTbThreads - 1) / kTbThreads;
    for (int it0 = 0; it0 < iters; it0 += kTbChunk) {
        const int vb = v0 + it0 * kTbThreads + (int)threadIdx.x;
        int hv[kTbChunk];
        float xv[kTbChunk];
        #pragma unroll
        for (int u = 0; u < kTbChunk; ++u) {
            const int v = min(vb + u * kTbThreads, v1 - 1);
            hv[u] = H > 0 ? hot_index[v] : -1;
            xv[u] = l[v];
        }
        #pragma unroll
        for (int u = 0; u < kTbChunk; ++u) {     // outside, or hot (handled per node): unused
            const bool use = vb + u * kTbThreads < v1 && !(hv[u] >= 0 && hv[u] < H);
            xv[u] = use ? xv[u] : -__builtin_huge_valf();
        }
        fold_chunk(xv, [&](int u) { return vb + u * kTbThreads; }, k, lane, s_exp2, os, tk);
    }
    block_reduce_part(os, tk, k, rows + (size_t)row * gridDim.y + seg, s_exp2);
    // this row's logits of the hot tokens, contiguous for the per-node passes
    if (H > 0) {
        const int c_len = (H + gridDim.y - 1) / gridDim.y;
        const int c0 = seg * c_len, c1 = min(H, c0 + c_len);
        float *lh = hot_logits + (size_t)row * H;
        constexpr int kG = 8;                        // gathers per thread in flight together
        for (int cb = c0 + (int)threadIdx.x; cb < c1; cb += kG * kTbThreads) {
            int hv[kG];
            float hx[kG];
            #pragma unroll
            for (int u = 0; u < kG; ++u) {
                const int c = cb + u * kTbThreads;
                hv[u] = c < c1 ? hot_vocab[c] : -1;
            }
            #pragma unroll
            for (int u = 0; u < kG; ++u) hx[u] = (hv[u] >= 0 && hv[u] < V) ? l[hv[u]] : -__builtin_huge_valf();
            #pragma unroll
            for (int u = 0; u < kG; ++u)
                if (cb + u * kTbThreads < c1) lh[cb + u * kTbThreads] = hx[u];
        }
    }
    if (seg == 0 && row % S == 0 && threadIdx.x == 0) {
        const int b = row / S;
        node_tok[(size_t)b * max_nodes] = root_token[b];
        node_par[(size_t)b * max_nodes] = -1;
        node_joint[(size_t)b * max_nodes] = 1.0;
        const int t = root_token[b];
        TbFrontier *fr = frontier + b;
        fr->count = tb_window(accept_len, b, S, r).count > 0 ? 1 : 0;
        fr->slot[0] = TbSlot{0, t, hot_row(hot_index, t, V, H), 0, 1.0};
    }
}

// Hot columns of step i for frontier slot j of sequence b, one chunk of the
// columns per workgroup: x = l_i[hot[c]] + table[row of the node's token][c].
__global__ __launch_bounds__(kExpThreads) void tb_expand_kernel(
    const float *__restrict__ hot_logits, const uint16_t *__restrict__ table,
    const int32_t *__restrict__ hot_vocab, const int32_t *__restrict__ accept_len, int r, int S,
    int V, int H, int k, int step, int chunk_len, const TbFrontier *__restrict__ frontier,
    TbPart *__restrict__ parts) {
    const int b = blockIdx.x, j = blockIdx.y, c = blockIdx.z;
    const TbFrontier *fr = frontier + b;
    TbPart *out = parts + ((size_t)b * k + j) * gridDim.z + c;
    const int count = fr->count;
    const int h = fr->slot[j].h;                   // loaded with the count (j < kTbMaxK)
    const TbWindow win = tb_window(accept_len, b, S, r);
    if (step >= win.count) return;                 // this sequence's tree is complete
    if (j >= count) return;                        // no such frontier node at this step
    __shared__ double s_exp2[32];
    fill_exp2_table(s_exp2);
    __syncthreads();
    const float *lh = hot_logits + ((size_t)b * S + win.first + step) * H;
    const uint16_t *trow = table + (size_t)max(h, 0) * H;   // row 0 stands in when h < 0 (unused)
    const int c0 = c * chunk_len, c1 = min(H, c0 + chunk_len);
    OnlineSum os;
    WaveTopK tk;
    const int lane = threadIdx.x & (kWave - 1);
    const int iters = (max(c1 - c0, 0) + kExpThreads - 1) / kExpThreads;   // chunks as above
    for (int it0 = 0; it0 < iters; it0 += kTbChunk) {
        const int cb = c0 + it0 * kExpThreads + (int)threadIdx.x;
        // a full chunk needs no per-candidate range tests (kept out of the
        // common path: they cost registers and instructions)
        auto chunk = [&](auto full) {
            int vv[kTbChunk];
            float xv[kTbChunk];
            unsigned int rv[kTbChunk];
            if constexpr (full) {
                // four consecutive columns per lane and load (16-byte loads of
                // the logits and ids, 8-byte loads of the table entries)
                const int cq = c0 + it0 * kExpThreads + 4 * lane;
                #pragma unroll
                for (int q = 0; q < kTbChunk / 4; ++q) {
                    const int cc = cq + q * 4 * kExpThreads;
                    const i32x4 v4 = *reinterpret_cast<const i32x4 *>(hot_vocab + cc);
                    const f32x4 x4 = *reinterpret_cast<const f32x4 *>(lh + cc);
                    const u16x4 t4 = *reinterpret_cast<const u16x4 *>(trow + cc);
                    #pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        vv[4 * q + r] = v4[r];
                        xv[4 * q + r] = x4[r];
                        rv[4 * q + r] = t4[r];
                    }
                }
            } else {
                #pragma unroll
                for (int u = 0; u < kTbChunk; ++u) {
                    const int cc = min(cb + u * kExpThreads, c1 - 1);
                    vv[u] = hot_vocab[cc];
                    xv[u] = lh[cc];
                    rv[u] = trow[cc];
                }
            }
            #pragma unroll
            for (int u = 0; u < kTbChunk; ++u) {
                if (h >= 0) xv[u] += __uint_as_float(rv[u] << 16);
                const bool use = (full || cb + u * kExpThreads < c1) && (unsigned int)vv[u] < (unsigned int)V;
                xv[u] = use ? xv[u] : -__builtin_huge_valf();
            }
            fold_chunk(xv, [&](int u) { return vv[u]; }, k, lane, s_exp2, os, tk);
        };
        // full: every column of the chunk exists, and rows, chunk start, the
        // caller's arrays and the workspace row are aligned for the wide loads
        if (c1 - (c0 + it0 * kExpThreads) >= kTbChunk * kExpThreads && (H & 3) == 0 && (c0 & 3) == 0 &&
            (reinterpret_cast<uintptr_t>(hot_vocab) & 15) == 0 && (reinterpret_cast<uintptr_t>(table) & 7) == 0 &&
            (reinterpret_cast<uintptr_t>(lh) & 15) == 0)
            chunk(std::true_type{});
        else
            chunk(std::false_type{});
    }
    wave_reduce_part(os, tk, k, lane, out, s_exp2);
}

// One workgroup per sequence, one wave per frontier node of step i: combine the
// step's row partials with the node's column partials (all loaded at once)
// into its k children (token, probability, joint probability), then choose
// the next frontier.
template <int CPL>          // candidate keys per lane: (segs + chunks) * k <= 64 * CPL
__global__ __launch_bounds__(kTbMaxK * kWave) void tb_select_kernel(
    const TbPart *__restrict__ rows, int segs, const TbPart *__restrict__ parts, int chunks,
    const int32_t *__restrict__ accept_len, const int32_t *__restrict__ hot_index, int r, int S,
    int V, int H, int k, int step, int max_nodes, int32_t *__restrict__ node_tok,
    int32_t *__restrict__ node_par, double *__restrict__ node_joint,
    TbFrontier *__restrict__ frontier) {
    constexpr int kCandPerLane = CPL;
    __shared__ double s_joint[kTbMaxK * kTbMaxK];
    __shared__ int s_tok[kTbMaxK * kTbMaxK];
    __shared__ int s_hot[kTbMaxK * kTbMaxK];
    const int b = blockIdx.x;
    const int lane = threadIdx.x & (kWave - 1), j = threadIdx.x / kWave;
    const TbWindow win = tb_window(accept_len, b, S, r);
    if (step >= win.count) return;                 // uniform: this sequence is done
    TbFrontier *fr = frontier + b;
    const int nf = fr->count;
    // nodes before this step: the root, then k children per frontier node of
    // every earlier step (1 at step 0, k afterwards)
    const int base = step == 0 ? 1 : 1 + k + (step - 1) * k * k;
    if (j < nf) {
        const TbPart *rp = rows + ((size_t)b * S + win.first + step) * segs;
        const TbPart *cp = parts + ((size_t)b * k + j) * chunks;
        const int nparts = segs + chunks;
        const int ncand = nparts * k;
        const TbSlot sl = fr->slot[j];
        const int f = sl.node;
        // every load of this node is issued before any is used
        float pm = -__builtin_huge_valf();
        double ps = 0.0;
        if (lane < nparts) {
            const TbPart *pp = lane < segs ? rp + lane : cp + (lane - segs);
            pm = pp->m;
            ps = pp->s;
        }
        unsigned long long cand[kCandPerLane];
        #pragma unroll
        for (int u = 0; u < kCandPerLane; ++u) {
            const int idx = lane + u * kWave;
            unsigned long long key = 0ull;
            if (idx < ncand) {
                const int q = idx / k, r = idx - q * k;
                key = q < segs ? rp[q].key[r] : cp[q - segs].key[r];
            }
            cand[u] = key;
        }
        const double pj = sl.joint;
        const float m = wave_allmax(pm);
        const double s = wave_allsum(pm == -__builtin_huge_valf() ? 0.0 : ps * exp((double)pm - (double)m));
        // rank r's key goes to lane r; the children's probabilities are then
        // computed by lanes 0..k-1 at once
        unsigned long long mine = 0ull;
        for (int r = 0; r < k; ++r) {
            unsigned long long best = 0ull;
            #pragma unroll
            for (int u = 0; u < kCandPerLane; ++u) best = umax64(best, cand[u]);
            best = wave_max64(best);
            #pragma unroll
            for (int u = 0; u < kCandPerLane; ++u) cand[u] = cand[u] == best ? 0ull : cand[u];
            mine = lane == r ? best : mine;
        }
        if (lane < k) {
            const size_t at = (size_t)b * max_nodes + base + j * k + lane;
            double joint = 0.0;
            int tok = -1;
            if (mine != 0ull) {
                tok = key_index(mine);
                joint = pj * (exp((double)key_value(mine) - (double)m) / s);
            }
            node_tok[at] = tok;
            node_par[at] = f;
            node_joint[at] = joint;
            s_joint[j * k + lane] = joint;
            s_tok[j * k + lane] = tok;
            s_hot[j * k + lane] = hot_row(hot_index, tok, V, H);   // loaded now, used after the ranking
        }
    }
    __syncthreads();
    // next frontier: the k children of this step with the largest joint
    // probabilities, largest first, ties to the earlier child. Child i's rank
    // is the number of children before it in that order.
    // tpc threads share child i's count (consecutive lanes, nc * tpc <= the
    // workgroup's threads), then add their parts.
    const int nc = nf * k;
    int tpc = 16;
    while (tpc > 1 && nc * tpc > kTbMaxK * kWave) tpc >>= 1;
    {
        const int i = threadIdx.x / tpc, part = threadIdx.x % tpc;
        int rank = 0;
        double ji = 0.0;
        if (i < nc) {
            ji = s_joint[i];
            for (int q = part; q < nc; q += tpc) {
                const double jq = s_joint[q];
                rank += (jq > ji || (jq == ji && q < i)) ? 1 : 0;
            }
        }
        rank = group_sum(rank, tpc);
        if (i < nc && part == 0 && rank < k)
            fr->slot[rank] = TbSlot{base + i, s_tok[i], s_hot[i], 0, ji};
    }
    if (threadIdx.x == 0) fr->count = min(k, nc);
}

// One workgroup per sequence: keep the `budget` nodes of largest joint
// probability (ties to the earlier node), in creation order, parents renumbered.
__global__ __launch_bounds__(kPruneThreads) void tb_prune_kernel(
    const int32_t *__restrict__ accept_len, int r, int S, int k, int budget, int max_nodes,
    const int32_t *__restrict__ node_tok,
    const int32_t *__restrict__ node_par, const double *__restrict__ node_joint,
    int32_t *__restrict__ parent, int32_t *__restrict__ token, float *__restrict__ joint,
    int32_t *__restrict__ num_nodes) {
    __shared__ double s_j[kPruneSlots];
    __shared__ short s_i[kPruneSlots];
    __shared__ short s_new[kPruneSlots];
    __shared__ int s_warp[kPruneThreads / kWave];
    const int b = blockIdx.x, tid = threadIdx.x;
    const size_t nb = (size_t)b * max_nodes;
    const TbWindow win = tb_window(accept_len, b, S, r);
    const int n = win.count < 0 ? 0 : win.count == 0 ? 1 : 1 + k + (win.count - 1) * k * k;
    int P2 = 1;
    while (P2 < n) P2 <<= 1;
    for (int i = tid; i < P2; i += kPruneThreads) {
        s_j[i] = i < n ? node_joint[nb + i] : -1.0;
        s_i[i] = (short)i;
    }
    __syncthreads();
    // bitonic sort: joint descending, index ascending
    for (int size = 2; size <= P2; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = tid; i < P2; i += kPruneThreads) {
                const int pr = i ^ stride;
                if (pr > i) {
                    const bool desc = (i & size) == 0;
                    const double ja = s_j[i], jb = s_j[pr];
                    const int ia = s_i[i], ib = s_i[pr];
                    const bool a_first = ja > jb || (ja == jb && ia < ib);
                    if (a_first != desc) {
                        s_j[i] = jb; s_j[pr] = ja;
                        s_i[i] = (short)ib; s_i[pr] = (short)ia;
                    }
                }
            }
            __syncthreads();
        }
    }
    // keep flags by creation index, then ranks in creation order
    const int kept = min(budget, n);
    for (int i = tid; i < kPruneSlots; i += kPruneThreads) s_new[i] = 0;
    __syncthreads();
    for (int i = tid; i < kept; i += kPruneThreads) s_new[s_i[i]] = 1;
    __syncthreads();
    // exclusive prefix count of the flags (n <= 4096: 4 per thread)
    constexpr int kPer = kPruneSlots / kPruneThreads;
    int f[kPer], run = 0;
    #pragma unroll
    for (int u = 0; u < kPer; ++u) { f[u] = s_new[tid * kPer + u]; run += f[u]; }
    const int lane = tid & (kWave - 1), w = tid / kWave;
    int incl = run;
    #pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int o = __shfl_up(incl, off);
        if (lane >= off) incl += o;
    }
    if (lane == kWave - 1) s_warp[w] = incl;
    __syncthreads();
    int before = incl - run;
    for (int q = 0; q < w; ++q) before += s_warp[q];
    __syncthreads();
    #pragma unroll
    for (int u = 0; u < kPer; ++u) {
        const int i = tid * kPer + u;
        s_new[i] = f[u] ? (short)before : (short)-1;
        before += f[u];
    }
    __syncthreads();
    for (int i = tid; i < n; i += kPruneThreads) {
        const int ni = s_new[i];
        if (ni < 0) continue;
        const int pp = node_par[nb + i];
        parent[(size_t)b * budget + ni] = pp < 0 ? -1 : s_new[pp];
        token[(size_t)b * budget + ni] = node_tok[nb + i];
        joint[(size_t)b * budget + ni] = (float)node_joint[nb + i];
    }
    for (int i = kept + tid; i < budget; i += kPruneThreads) {
        parent[(size_t)b * budget + i] = -1;
        token[(size_t)b * budget + i] = -1;
        joint[(size_t)b * budget + i] = 0.f;
    }
    if (tid == 0) num_nodes[b] = kept;
}

}  // namespace

TreeBuildPlan tree_build_plan(int B, int S, int V, int H, int k) {
    TreeBuildPlan pl;
    const long rows = (long)B * S;
    // at least 16384 tokens per workgroup (64 per thread), so that the top-k
    // filter, not the insertions, sets the cost per token
    long segs = ((long)V + 16383) / 16384;
    if (segs > 32) segs = 32;
    if (segs < 1) segs = 1;
    pl.segs = (int)segs;
    pl.seg_len = (int)(((long)V + segs - 1) / segs);
    long chunks = 0;
    if (H > 0) {
        chunks = ((long)H + 2047) / 2048;            // at least 2048 columns per (one-wave) workgroup
        if (chunks > 32) chunks = 32;
        if (chunks < 1) chunks = 1;
    }
    pl.chunks = (int)chunks;
    pl.chunk_len = chunks > 0 ? (int)(((long)H + chunks - 1) / chunks) : 0;
    pl.max_nodes = 1 + k + (S - 1) * k * k;
    pl.rows_bytes = (size_t)rows * segs * sizeof(TbPart);
    pl.hot_logits_bytes = (size_t)rows * H * sizeof(float);
    pl.parts_bytes = (size_t)B * k * (chunks > 0 ? chunks : 1) * sizeof(TbPart);
    pl.nodes_bytes = (size_t)B * pl.max_nodes * (2 * sizeof(int32_t) + sizeof(double));
    pl.frontier_bytes = (size_t)B * sizeof(TbFrontier);
    return pl;
}

hipError_t launch_tree_build(const float *logits, const int32_t *root_token,
                             const uint16_t *table, const int32_t *hot_vocab,
                             const int32_t *hot_index, const int32_t *accept_len, int r, int B,
                             int S, int V, int H, int k, int budget, int32_t *parent,
                             int32_t *token, float *joint, int32_t *num_nodes, void *workspace,
                             hipStream_t s) {
    if (B == 0) return hipSuccess;
    const TreeBuildPlan pl = tree_build_plan(B, S, V, H, k);
    char *base = static_cast<char *>(workspace);
    auto carve = [&](size_t bytes) {
        char *p = base;
        base += (bytes + 255) & ~(size_t)255;
        return p;
    };
    TbPart *rows = reinterpret_cast<TbPart *>(carve(pl.rows_bytes));
    TbPart *parts = reinterpret_cast<TbPart *>(carve(pl.parts_bytes));
    float *hot_logits = reinterpret_cast<float *>(carve(pl.hot_logits_bytes));
    const size_t nn = (size_t)B * pl.max_nodes;
    int32_t *node_tok = reinterpret_cast<int32_t *>(carve(nn * sizeof(int32_t)));
    int32_t *node_par = reinterpret_cast<int32_t *>(carve(nn * sizeof(int32_t)));
    double *node_joint = reinterpret_cast<double *>(carve(nn * sizeof(double)));
    TbFrontier *frontier = reinterpret_cast<TbFrontier *>(carve(pl.frontier_bytes));

    hipError_t e = launch_kernel(tb_rows_kernel, dim3(B * S, pl.segs), dim3(kTbThreads), s, logits,
                                 hot_vocab, hot_index, root_token, accept_len, r, S, V, H, k,
                                 pl.seg_len, rows, hot_logits, pl.max_nodes, node_tok, node_par,
                                 node_joint, frontier);
    for (int i = 0; i < S && e == hipSuccess; ++i) {
        if (pl.chunks > 0)
            e = launch_kernel(tb_expand_kernel, dim3(B, k, pl.chunks), dim3(kExpThreads), s,
                              hot_logits, table, hot_vocab, accept_len, r, S, V, H, k, i,
                              pl.chunk_len, (const TbFrontier *)frontier, parts);
        if (e == hipSuccess) {
            // candidate keys per lane of the selection: (segs + chunks) k of them
            const int ncand = (pl.segs + pl.chunks) * k;
            auto sel = ncand <= 2 * kWave ? tb_select_kernel<2>
                       : ncand <= 4 * kWave ? tb_select_kernel<4>
                       : ncand <= 8 * kWave ? tb_select_kernel<8> : tb_select_kernel<16>;
            e = launch_kernel(sel, dim3(B), dim3(kTbMaxK * kWave), s, rows, pl.segs, parts,
                              pl.chunks, accept_len, hot_index, r, S, V, H, k, i, pl.max_nodes,
                              node_tok, node_par, node_joint, frontier);
        }
    }
    if (e == hipSuccess)
        e = launch_kernel(tb_prune_kernel, dim3(B), dim3(kPruneThreads), s, accept_len, r, S, k,
                          budget, pl.max_nodes, node_tok, node_par, node_joint, parent, token,
                          joint, num_nodes);
    return e;
}

}  // namespace tv
