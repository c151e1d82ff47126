// Greedy verification for gfx950: per-node vocabulary argmax, then the longest
// accepted root path and the bonus token (§5.3; §7.1 decodes at temperature 0).
//
// Kernel 1 streams the fp32 logits once (the step's largest HBM read). Each
// workgroup reduces one contiguous segment of one row to a single 64-bit key
// that orders candidates exactly like the definition: larger value first
// (NaN above everything, -0 folded onto +0), then lower index. Rows are cut
// into enough segments to give the launch a few thousand workgroups, so even
// a batch of a handful of rows fills every CU.
//
// Kernel 2 runs one workgroup per sequence: thread i folds node i's segment
// keys into its argmax, then marks the node accepted when every edge of its
// root path matches, and a block reduction picks the deepest accepted node
// (lowest index on ties) whose path and argmax give the outputs.
//
// Ragged batches (a verification-fusion forest per sequence, §6.2): nodes at
// or past num_nodes[b] are padding. Their logits rows are not streamed, their
// argmax is -1 and they take no part in acceptance; a sequence without nodes
// accepts nothing (length 0, bonus -1).
#include "tv_internal.h"

namespace tv {
namespace {

constexpr int kArgmaxThreads = 256;
constexpr int kAcceptThreads = 256;

__device__ __forceinline__ unsigned long long umax64(unsigned long long a, unsigned long long b) {
    return a > b ? a : b;
}

__device__ __forceinline__ int node_count(const int32_t *num_nodes, int b, int N) {
    if (!num_nodes) return N;
    const int n = num_nodes[b];
    return n < 0 ? 0 : (n > N ? N : n);
}

__device__ __forceinline__ unsigned long long wave_max64(unsigned long long v) {
    #pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const unsigned int lo = __shfl_xor((unsigned int)v, off);
        const unsigned int hi = __shfl_xor((unsigned int)(v >> 32), off);
        v = umax64(v, ((unsigned long long)hi << 32) | lo);
    }
    return v;
}

// One workgroup per (row, segment). seg_len is a multiple of 4.
__global__ __launch_bounds__(kArgmaxThreads) void argmax_segments_kernel(
    const float *__restrict__ logits, const int32_t *__restrict__ num_nodes, int N, int V,
    int segs, int seg_len, unsigned long long *__restrict__ ws) {
    const size_t row = blockIdx.x;
    const int seg = blockIdx.y;
    if (num_nodes && (int)(row % N) >= node_count(num_nodes, (int)(row / N), N)) {
        if (threadIdx.x == 0) ws[row * segs + seg] = 0ull;     // padding node: nothing read
        return;
    }
    const int v0 = seg * seg_len;
    const int v1 = min(V, v0 + seg_len);
    const float *x = logits + row * (size_t)V;
    unsigned long long best = 0ull;      // below every real key
    const int tid = threadIdx.x;

    // Vector path when the row start is 16-byte aligned; a scalar head/tail otherwise.
    const uintptr_t addr = reinterpret_cast<uintptr_t>(x + v0);
    const int head = (int)(((16 - (addr & 15)) & 15) / 4);
    const int vh = min(v1, v0 + head);
    for (int v = v0 + tid; v < vh; v += kArgmaxThreads)
        best = umax64(best, pack_key(order_key(x[v]), (unsigned int)v));
    const int nvec = (v1 - vh) / 4;
    const f32x4 *xv = reinterpret_cast<const f32x4 *>(x + vh);
    constexpr int U = 4;
    int i = tid;
    for (; i + (U - 1) * kArgmaxThreads < nvec; i += U * kArgmaxThreads) {
        f32x4 r[U];
        #pragma unroll
        for (int u = 0; u < U; ++u) r[u] = __builtin_nontemporal_load(xv + i + u * kArgmaxThreads);
        #pragma unroll
        for (int u = 0; u < U; ++u) {
            const unsigned int base = (unsigned int)(vh + 4 * (i + u * kArgmaxThreads));
            #pragma unroll
            for (int k = 0; k < 4; ++k) best = umax64(best, pack_key(order_key(r[u][k]), base + k));
        }
    }
    for (; i < nvec; i += kArgmaxThreads) {
        const f32x4 r = __builtin_nontemporal_load(xv + i);
        const unsigned int base = (unsigned int)(vh + 4 * i);
        #pragma unroll
        for (int k = 0; k < 4; ++k) best = umax64(best, pack_key(order_key(r[k]), base + k));
    }
    for (int v = vh + 4 * nvec + tid; v < v1; v += kArgmaxThreads)
        best = umax64(best, pack_key(order_key(x[v]), (unsigned int)v));

    best = wave_max64(best);
    __shared__ unsigned long long part[kArgmaxThreads / kWave];
    if ((tid & (kWave - 1)) == 0) part[tid / kWave] = best;
    __syncthreads();
    if (tid == 0) {
        unsigned long long m = part[0];
        #pragma unroll
        for (int k = 1; k < kArgmaxThreads / kWave; ++k) m = umax64(m, part[k]);
        ws[row * segs + seg] = m;
    }
}

__global__ __launch_bounds__(kAcceptThreads) void accept_kernel(
    const unsigned long long *__restrict__ ws, int segs, const int32_t *__restrict__ draft,
    const int32_t *__restrict__ parent, const int32_t *__restrict__ num_nodes, int N,
    int32_t *__restrict__ argmax_out, int32_t *__restrict__ accept_len,
    int32_t *__restrict__ accept_idx, int32_t *__restrict__ bonus) {
    const int b = blockIdx.x;
    const int i = threadIdx.x;
    const int nb = node_count(num_nodes, b, N);
    __shared__ int s_par[kMaxNodes];
    __shared__ int s_amax[kMaxNodes];
    __shared__ int s_match[kMaxNodes];
    __shared__ unsigned int s_best[kAcceptThreads / kWave];

    if (i < nb) {
        const size_t row = (size_t)b * N + i;
        unsigned long long m = 0ull;
        for (int s = 0; s < segs; ++s) m = umax64(m, ws[row * segs + s]);
        const int am = (int)(0xFFFFFFFFu - (unsigned int)m);
        s_amax[i] = am;
        argmax_out[row] = am;
        int pi = parent[row];
        if (pi < -1 || pi >= i) pi = -1;                 // contract violation: treat as a root
        s_par[i] = pi;
        accept_idx[row] = -1;
    } else if (i < N) {
        const size_t row = (size_t)b * N + i;
        argmax_out[row] = -1;
        accept_idx[row] = -1;
    }
    __syncthreads();
    // an edge (parent -> i) matches when i's draft token is the parent's argmax
    if (i < nb) {
        const int pi = s_par[i];
        s_match[i] = (pi < 0) || (draft[(size_t)b * N + i] == s_amax[pi]);
    }
    __syncthreads();
    unsigned int key = 0u;              // (depth + 1) << 16 | (0xFFFF - i) for accepted nodes
    if (i < nb) {
        int ok = 1, depth = 0;
        for (int j = i; s_par[j] >= 0; j = s_par[j]) {
            ok &= s_match[j];
            ++depth;
        }
        if (ok) key = ((unsigned int)(depth + 1) << 16) | (0xFFFFu - (unsigned int)i);
    }
    #pragma unroll
    for (int off = 32; off > 0; off >>= 1) key = max(key, (unsigned int)__shfl_xor((int)key, off));
    if ((i & (kWave - 1)) == 0) s_best[i / kWave] = key;
    __syncthreads();
    if (i == 0) {
        unsigned int k = s_best[0];
        #pragma unroll
        for (int w = 1; w < kAcceptThreads / kWave; ++w) k = max(k, s_best[w]);
        const int sel = (int)(0xFFFFu - (k & 0xFFFFu));
        const int len = (int)(k >> 16);          // 0 when the sequence has no nodes
        accept_len[b] = len;
        bonus[b] = len > 0 ? s_amax[sel] : -1;
        int j = sel;
        for (int d = len - 1; d >= 0; --d) {
            accept_idx[(size_t)b * N + d] = j;
            j = s_par[j];
        }
    }
}

}  // namespace

hipError_t launch_argmax_accept(const float *logits, const int32_t *draft, const int32_t *parent,
                                const int32_t *num_nodes, int B, int N, int V, int segs,
                                int seg_len, int32_t *argmax_out,
                                int32_t *accept_len, int32_t *accept_idx, int32_t *bonus,
                                unsigned long long *ws, hipStream_t s) {
    if (B == 0) return hipSuccess;
    const hipError_t e = launch_kernel(argmax_segments_kernel, dim3(B * N, segs),
                                       dim3(kArgmaxThreads), s, logits, num_nodes, N, V, segs,
                                       seg_len, ws);
    if (e != hipSuccess) return e;
    return launch_accept(ws, segs, draft, parent, num_nodes, B, N, argmax_out, accept_len,
                         accept_idx, bonus, s);
}

hipError_t launch_accept(const unsigned long long *keys, int segs, const int32_t *draft,
                         const int32_t *parent, const int32_t *num_nodes, int B, int N,
                         int32_t *argmax_out, int32_t *accept_len, int32_t *accept_idx,
                         int32_t *bonus, hipStream_t s) {
    if (B == 0) return hipSuccess;
    return launch_kernel(accept_kernel, dim3(B), dim3(kAcceptThreads), s, keys, segs, draft,
                         parent, num_nodes, N, argmax_out, accept_len, accept_idx, bonus);
}

}  // namespace tv
