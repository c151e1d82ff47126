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

__device__ __forceinline__ unsigned long long umax64(unsigned long long a, unsigned long long b) {
    return a > b ? a : b;
}

__device__ __forceinline__ unsigned long long shfl_xor64(unsigned long long v, int off) {
    const unsigned int lo = __shfl_xor((unsigned int)v, off);
    const unsigned int hi = __shfl_xor((unsigned int)(v >> 32), off);
    return ((unsigned long long)hi << 32) | lo;
}

__device__ __forceinline__ float key_value(unsigned long long key) {
    const unsigned int k = (unsigned int)(key >> 32);
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

__device__ __forceinline__ int key_index(unsigned long long key) {
    return (int)(0xFFFFFFFFu - (unsigned int)key);
}

// Running (max, sum of exp(x - max)) of one thread, fp64 sums.
struct OnlineSum {
    float m = -__builtin_huge_valf();
    double s = 0.0;
    __device__ __forceinline__ void add(float x) {
        if (x == -__builtin_huge_valf()) return;        // contributes exp(-inf) = 0
        if (x > m) {
            s = (m == -__builtin_huge_valf()) ? 1.0 : s * exp((double)m - (double)x) + 1.0;
            m = x;
        } else {
            s += exp((double)x - (double)m);
        }
    }
    __device__ __forceinline__ void merge(float m2, double s2) {
        if (m2 == -__builtin_huge_valf()) return;
        if (m == -__builtin_huge_valf()) { m = m2; s = s2; return; }
        const float mn = fmaxf(m, m2);
        s = s * exp((double)m - (double)mn) + s2 * exp((double)m2 - (double)mn);
        m = mn;
    }
};

// Thread-local top-k list in registers, descending; k is a runtime value
// <= kTbMaxK and the list is handled with fixed indices only.
struct TopK {
    unsigned long long t[kTbMaxK];
    unsigned long long kmin;          // the k-th entry (0 while the list is not full)
    __device__ __forceinline__ void init() {
        #pragma unroll
        for (int j = 0; j < kTbMaxK; ++j) t[j] = 0ull;
        kmin = 0ull;
    }
    __device__ __forceinline__ void insert(unsigned long long key, int k) {
        if (key <= kmin) return;
        #pragma unroll
        for (int j = 0; j < kTbMaxK; ++j) {
            if (j < k && key > t[j]) {
                const unsigned long long tmp = t[j];
                t[j] = key;
                key = tmp;
            }
        }
        unsigned long long km = 0ull;
        #pragma unroll
        for (int j = 0; j < kTbMaxK; ++j) km = (j == k - 1) ? t[j] : km;
        kmin = km;
    }
    __device__ __forceinline__ void pop_front() {
        #pragma unroll
        for (int j = 0; j < kTbMaxK - 1; ++j) t[j] = t[j + 1];
        t[kTbMaxK - 1] = 0ull;
    }
};

// Workgroup reduction of every thread's (OnlineSum, TopK) into one TbPart.
__device__ void block_reduce_part(OnlineSum os, TopK &tk, int k, TbPart *out) {
    __shared__ float s_m[kTbWaves];
    __shared__ double s_s[kTbWaves];
    __shared__ unsigned long long s_key[kTbWaves];
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    // (max, sum)
    #pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const float m2 = __shfl_xor(os.m, off);
        const double s2 = __shfl_xor(os.s, off);
        os.merge(m2, s2);
    }
    if (lane == 0) { s_m[wave] = os.m; s_s[wave] = os.s; }
    __syncthreads();
    if (threadIdx.x == 0) {
        OnlineSum t;
        for (int w = 0; w < kTbWaves; ++w) t.merge(s_m[w], s_s[w]);
        out->m = t.m;
        out->pad = 0;
        out->s = t.s;
    }
    // top-k: k rounds, each takes the largest head and pops it from its owner
    for (int r = 0; r < k; ++r) {
        unsigned long long best = tk.t[0];
        #pragma unroll
        for (int off = 32; off > 0; off >>= 1) best = umax64(best, shfl_xor64(best, off));
        __syncthreads();                         // s_key of the previous round is consumed
        if (lane == 0) s_key[wave] = best;
        __syncthreads();
        unsigned long long top = s_key[0];
        #pragma unroll
        for (int w = 1; w < kTbWaves; ++w) top = umax64(top, s_key[w]);
        if (top != 0ull && tk.t[0] == top) tk.pop_front();
        if (threadIdx.x == 0) out->key[r] = top;
    }
    if (threadIdx.x == 0)
        for (int r = k; r < kTbMaxK; ++r) out->key[r] = 0ull;
}

// Node-independent part of every (sequence, step): the non-hot tokens of the
// step's logits, one segment of the vocabulary per workgroup. Workgroup
// (row (b, 0), segment 0) also places the root and the first frontier.
__global__ __launch_bounds__(kTbThreads) void tb_rows_kernel(
    const float *__restrict__ logits, const int32_t *__restrict__ hot_index,
    const int32_t *__restrict__ root_token, int S, int V, int H, int k, int seg_len,
    TbPart *__restrict__ rows, int max_nodes, int32_t *__restrict__ node_tok,
    int32_t *__restrict__ node_par, double *__restrict__ node_joint,
    int32_t *__restrict__ frontier) {
    const int row = blockIdx.x, seg = blockIdx.y;
    const int v0 = seg * seg_len, v1 = min(V, v0 + seg_len);
    const float *l = logits + (size_t)row * V;
    OnlineSum os;
    TopK tk;
    tk.init();
    for (int v = v0 + threadIdx.x; v < v1; v += kTbThreads) {
        const int h = H > 0 ? hot_index[v] : -1;
        if (h >= 0 && h < H) continue;             // hot: handled per frontier node
        const float x = l[v];
        os.add(x);
        tk.insert(pack_key(order_key(x), (unsigned int)v), k);
    }
    block_reduce_part(os, tk, k, rows + (size_t)row * gridDim.y + seg);
    if (seg == 0 && row % S == 0 && threadIdx.x == 0) {
        const int b = row / S;
        node_tok[(size_t)b * max_nodes] = root_token[b];
        node_par[(size_t)b * max_nodes] = -1;
        node_joint[(size_t)b * max_nodes] = 1.0;
        frontier[b * (kTbMaxK + 1)] = 1;           // count, then node ids
        frontier[b * (kTbMaxK + 1) + 1] = 0;
    }
}

// Hot columns of step i for frontier slot j of sequence b, one chunk of the
// columns per workgroup: x = l_i[hot[c]] + table[row of the node's token][c].
__global__ __launch_bounds__(kTbThreads) void tb_expand_kernel(
    const float *__restrict__ logits, const uint16_t *__restrict__ table,
    const int32_t *__restrict__ hot_vocab, const int32_t *__restrict__ hot_index, int S, int V,
    int H, int k, int step, int chunk_len, const int32_t *__restrict__ node_tok, int max_nodes,
    const int32_t *__restrict__ frontier, TbPart *__restrict__ parts) {
    const int b = blockIdx.x, j = blockIdx.y, c = blockIdx.z;
    const int *fr = frontier + b * (kTbMaxK + 1);
    TbPart *out = parts + ((size_t)b * k + j) * gridDim.z + c;
    if (j >= fr[0]) return;                        // no such frontier node at this step
    const int t = node_tok[(size_t)b * max_nodes + fr[1 + j]];
    int h = (t >= 0 && t < V) ? hot_index[t] : -1;
    if (h >= H) h = -1;
    const float *l = logits + ((size_t)b * S + step) * V;
    const uint16_t *r = h >= 0 ? table + (size_t)h * H : nullptr;
    const int c0 = c * chunk_len, c1 = min(H, c0 + chunk_len);
    OnlineSum os;
    TopK tk;
    tk.init();
    for (int cc = c0 + threadIdx.x; cc < c1; cc += kTbThreads) {
        const int v = hot_vocab[cc];
        if (v < 0 || v >= V) continue;
        float x = l[v];
        if (r) x += __uint_as_float((unsigned int)r[cc] << 16);
        os.add(x);
        tk.insert(pack_key(order_key(x), (unsigned int)v), k);
    }
    block_reduce_part(os, tk, k, out);
}

// One workgroup per sequence: for every frontier node of step i, combine the
// step's row partials with the node's column partials into its k children
// (token, probability, joint probability), then choose the next frontier.
__global__ __launch_bounds__(kTbThreads) void tb_select_kernel(
    const TbPart *__restrict__ rows, int segs, const TbPart *__restrict__ parts, int chunks,
    int S, int k, int step, int max_nodes, int32_t *__restrict__ node_tok,
    int32_t *__restrict__ node_par, double *__restrict__ node_joint,
    int32_t *__restrict__ frontier) {
    constexpr int kCandPerLane = 16;          // (segs + chunks) * k <= (32 + 32) * 16 candidates
    __shared__ double s_joint[kTbMaxK * kTbMaxK];
    const int b = blockIdx.x;
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    int *fr = frontier + b * (kTbMaxK + 1);
    const int nf = fr[0];
    // nodes before this step: the root, then k children per frontier node of
    // every earlier step (1 at step 0, k afterwards)
    const int base = step == 0 ? 1 : 1 + k + (step - 1) * k * k;
    const TbPart *rp = rows + ((size_t)b * S + step) * segs;
    const int nparts = segs + chunks;
    const int ncand = nparts * k;
    for (int j = wave; j < nf; j += kTbWaves) {
        const TbPart *cp = parts + ((size_t)b * k + j) * chunks;
        // max and denominator over all partials
        float m = -__builtin_huge_valf();
        for (int q = lane; q < nparts; q += kWave) m = fmaxf(m, q < segs ? rp[q].m : cp[q - segs].m);
        #pragma unroll
        for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
        double s = 0.0;
        for (int q = lane; q < nparts; q += kWave) {
            const TbPart &pp = q < segs ? rp[q] : cp[q - segs];
            if (pp.m != -__builtin_huge_valf()) s += pp.s * exp((double)pp.m - (double)m);
        }
        #pragma unroll
        for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
        // top-k of all candidate keys
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
        const int f = fr[1 + j];
        const double pj = node_joint[(size_t)b * max_nodes + f];
        for (int r = 0; r < k; ++r) {
            unsigned long long best = 0ull;
            #pragma unroll
            for (int u = 0; u < kCandPerLane; ++u) best = umax64(best, cand[u]);
            #pragma unroll
            for (int off = 32; off > 0; off >>= 1) best = umax64(best, shfl_xor64(best, off));
            #pragma unroll
            for (int u = 0; u < kCandPerLane; ++u) cand[u] = cand[u] == best ? 0ull : cand[u];
            if (lane == 0) {
                const int n = base + j * k + r;
                const size_t at = (size_t)b * max_nodes + n;
                double joint = 0.0;
                int tok = -1;
                if (best != 0ull) {
                    tok = key_index(best);
                    joint = pj * (exp((double)key_value(best) - (double)m) / s);
                }
                node_tok[at] = tok;
                node_par[at] = f;
                node_joint[at] = joint;
                s_joint[j * k + r] = joint;
            }
        }
    }
    __syncthreads();
    // next frontier: the k children of this step with the largest joint
    // probabilities, largest first, ties to the earlier child
    if (wave == 0) {
        const int nc = nf * k;
        int taken[4] = {0, 0, 0, 0};
        for (int r = 0; r < k && r < nc; ++r) {
            double bj = -1.0;
            int bi = 1 << 30;
            #pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = lane + u * kWave;
                if (i < nc && !taken[u]) {
                    const double jv = s_joint[i];
                    if (jv > bj || (jv == bj && i < bi)) { bj = jv; bi = i; }
                }
            }
            #pragma unroll
            for (int off = 32; off > 0; off >>= 1) {
                const double oj = __shfl_xor(bj, off);
                const int oi = __shfl_xor(bi, off);
                if (oj > bj || (oj == bj && oi < bi)) { bj = oj; bi = oi; }
            }
            #pragma unroll
            for (int u = 0; u < 4; ++u)
                if (lane + u * kWave == bi) taken[u] = 1;
            if (lane == 0) fr[1 + r] = base + bi;
        }
        if (lane == 0) fr[0] = min(k, nc);
    }
}

// One workgroup per sequence: keep the `budget` nodes of largest joint
// probability (ties to the earlier node), in creation order, parents renumbered.
__global__ __launch_bounds__(kPruneThreads) void tb_prune_kernel(
    int n, int budget, int max_nodes, const int32_t *__restrict__ node_tok,
    const int32_t *__restrict__ node_par, const double *__restrict__ node_joint,
    int32_t *__restrict__ parent, int32_t *__restrict__ token, float *__restrict__ joint,
    int32_t *__restrict__ num_nodes) {
    __shared__ double s_j[kPruneSlots];
    __shared__ short s_i[kPruneSlots];
    __shared__ short s_new[kPruneSlots];
    __shared__ int s_warp[kPruneThreads / kWave];
    const int b = blockIdx.x, tid = threadIdx.x;
    const size_t nb = (size_t)b * max_nodes;
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
    long segs = rows > 0 ? (2048 + rows - 1) / rows : 1;
    const long max_segs = ((long)V + 2047) / 2048;
    if (segs > max_segs) segs = max_segs;
    if (segs > 32) segs = 32;
    if (segs < 1) segs = 1;
    pl.segs = (int)segs;
    pl.seg_len = (int)(((long)V + segs - 1) / segs);
    long chunks = 0;
    if (H > 0) {
        const long slots = (long)B * k;
        chunks = slots > 0 ? (1024 + slots - 1) / slots : 1;
        const long max_chunks = ((long)H + 255) / 256;
        if (chunks > max_chunks) chunks = max_chunks;
        if (chunks > 32) chunks = 32;
        if (chunks < 1) chunks = 1;
    }
    pl.chunks = (int)chunks;
    pl.chunk_len = chunks > 0 ? (int)(((long)H + chunks - 1) / chunks) : 0;
    pl.max_nodes = 1 + k + (S - 1) * k * k;
    pl.rows_bytes = (size_t)rows * segs * sizeof(TbPart);
    pl.parts_bytes = (size_t)B * k * (chunks > 0 ? chunks : 1) * sizeof(TbPart);
    pl.nodes_bytes = (size_t)B * pl.max_nodes * (2 * sizeof(int32_t) + sizeof(double));
    pl.frontier_bytes = (size_t)B * (kTbMaxK + 1) * sizeof(int32_t);
    return pl;
}

hipError_t launch_tree_build(const float *logits, const int32_t *root_token,
                             const uint16_t *table, const int32_t *hot_vocab,
                             const int32_t *hot_index, int B, int S, int V, int H, int k,
                             int budget, int32_t *parent, int32_t *token, float *joint,
                             int32_t *num_nodes, void *workspace, hipStream_t s) {
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
    const size_t nn = (size_t)B * pl.max_nodes;
    int32_t *node_tok = reinterpret_cast<int32_t *>(carve(nn * sizeof(int32_t)));
    int32_t *node_par = reinterpret_cast<int32_t *>(carve(nn * sizeof(int32_t)));
    double *node_joint = reinterpret_cast<double *>(carve(nn * sizeof(double)));
    int32_t *frontier = reinterpret_cast<int32_t *>(carve(pl.frontier_bytes));

    hipError_t e = launch_kernel(tb_rows_kernel, dim3(B * S, pl.segs), dim3(kTbThreads), s, logits,
                                 hot_index, root_token, S, V, H, k, pl.seg_len, rows, pl.max_nodes,
                                 node_tok, node_par, node_joint, frontier);
    for (int i = 0; i < S && e == hipSuccess; ++i) {
        if (pl.chunks > 0)
            e = launch_kernel(tb_expand_kernel, dim3(B, k, pl.chunks), dim3(kTbThreads), s, logits,
                              table, hot_vocab, hot_index, S, V, H, k, i, pl.chunk_len, node_tok,
                              pl.max_nodes, frontier, parts);
        if (e == hipSuccess)
            e = launch_kernel(tb_select_kernel, dim3(B), dim3(kTbThreads), s, rows, pl.segs, parts,
                              pl.chunks, S, k, i, pl.max_nodes, node_tok, node_par, node_joint,
                              frontier);
    }
    if (e == hipSuccess)
        e = launch_kernel(tb_prune_kernel, dim3(B), dim3(kPruneThreads), s, pl.max_nodes, budget,
                          pl.max_nodes, node_tok, node_par, node_joint, parent, token, joint,
                          num_nodes);
    return e;
}

}  // namespace tv
