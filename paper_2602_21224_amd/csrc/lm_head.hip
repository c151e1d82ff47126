// LM head fused with the vocabulary argmax for gfx950: greedy verification
// without materialised logits.
//
// The target model's logit of tree node row r and vocabulary entry v is the
// dot product of the row's final hidden state with row v of the LM-head
// weight (the logits of many nodes are one matrix product, as the paper does
// on the draft side, §4.2), and greedy verification (§7.1: temperature 0;
// accepted path and bonus token, §5.3) needs only each row's argmax. This
// kernel computes hidden x W^T tile by tile on the matrix cores and reduces
// every tile straight to one 64-bit key per row, with the ordering of the
// stand-alone argmax (larger value first, NaN above everything, -0 == +0,
// lower id on ties), so the [rows, V] fp32 logits never exist in memory.
//
//   * Workgroup tile: 256 vocabulary entries (MFMA M) x 256 hidden rows
//     (MFMA N), the largest whose fp32 accumulators fit a CU's registers.
//     Eight waves (two per SIMD, so one wave's waits are covered by the
//     other's matrix work) in a 2 x 4 arrangement, each accumulating a
//     128 x 64 block in 8 v_mfma_f32_32x32x16_bf16 accumulators.
//   * Both operands are K-contiguous (W is [V, d], hidden is [R, d]), so both
//     stream into LDS the same way: global_load_lds_dwordx4 into a 4-stage
//     ring of 32-deep K slices. The four 16-byte chunks of each 64-byte row
//     slice are XOR-swizzled by bits 2-3 of the row, so the operand reads
//     (16 rows at one chunk per LDS pass) are free of bank conflicts.
//   * The reads of the next K step's operands and the loads of the slice
//     four ahead are interleaved one by one with the current step's MFMAs
//     (pinned by sched_barrier), and the ring hand-off (s_waitcnt vmcnt +
//     s_barrier) sits a few MFMAs into a slice's second K step, after this
//     wave's last read of the slice whose stage is refilled next: three
//     slices are in flight while one is computed.
//   * Workgroup order: ids are dispatched round-robin over the 8 XCDs, so
//     they are mapped such that the row blocks of one vocabulary tile run back
//     to back on one XCD and share its L2 copy of that weight tile.
//   * Epilogue: each lane folds its 64 values per row into a key, lanes l and
//     l ^ 32 combine, the two waves of a row block combine through LDS, and a
//     64-bit atomic maximum per (row, vocabulary tile) merges the tiles into
//     the row's key, which the greedy acceptance kernel then decodes.
#include "tv_internal.h"

namespace tv {
namespace {

#define LDS_AS __attribute__((address_space(3)))
#define GLOBAL_AS __attribute__((address_space(1)))

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;                              // two per SIMD
constexpr int kLmThreads = kWaves * kWave;
constexpr int kTileM = 256;                            // vocabulary entries per workgroup
constexpr int kTileN = 256;                            // hidden rows per workgroup
constexpr int kBK = 32;                                // K depth of one ring stage
constexpr int kStages = 4;                             // a power of two
constexpr int kSliceRow = kBK * 2;                     // bytes of one row's K slice
constexpr int kOperandBytes = kTileM * kSliceRow;      // 16 KB per operand per stage
constexpr int kStageBytes = 2 * kOperandBytes;         // W slice, then hidden slice
constexpr int kLoads = kOperandBytes / (kLmThreads * 16);   // 16-byte loads per operand per thread
constexpr int kWaveM = 128;                            // per-wave block: 2 waves along M
constexpr int kWaveN = kTileN / (kWaves / 2);
constexpr int kFragM = kWaveM / 32, kFragN = kWaveN / 32;
constexpr int kReads = kFragM + kFragN;                // fragment reads per K step
constexpr int kSteps = kFragM * kFragN;                // MFMAs per K step
static_assert(kTileM == kTileN, "both operands share one slice layout");
static_assert(kLoads * kWaves == 16, "one 1 KB block per load instruction: 16 blocks per operand");

__shared__ __attribute__((aligned(1024))) unsigned char g_lm_ring[kStages * kStageBytes];
__shared__ unsigned long long g_lm_keys[kWaves / 2][kWaveN];

__device__ __forceinline__ unsigned lds_addr(const void *p) {
    return (unsigned)(size_t)(const LDS_AS void *)p;
}

template <typename T>
__device__ __forceinline__ void tie(T &x) {
    asm volatile("" : "+v"(x));
}

__device__ __forceinline__ void lds_wait_all() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// s_waitcnt vmcnt(N) (gfx9 encoding: vmcnt in [3:0] and [15:14]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt is a 6-bit field");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ unsigned long long umax64(unsigned long long a, unsigned long long b) {
    return a > b ? a : b;
}

// Maximum of a 64-bit key held by lanes l and l ^ 32.
__device__ __forceinline__ unsigned long long halves_max64(unsigned long long x) {
    const unsigned lo = (unsigned)x, hi = (unsigned)(x >> 32);
    const auto l = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
    const auto h = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
    const unsigned long long a = ((unsigned long long)h[0] << 32) | l[0];
    const unsigned long long b = ((unsigned long long)h[1] << 32) | l[1];
    return umax64(a, b);
}

__global__ void lm_keys_clear_kernel(unsigned long long *__restrict__ keys, int R) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < R) keys[i] = 0ull;                  // below every real key
}

// grid: kNumXcd * ceil(vtiles / kNumXcd) * rblocks workgroups of kLmThreads threads.
__global__ __launch_bounds__(kLmThreads, 1) void lm_head_argmax_kernel(
    const uint16_t *__restrict__ hidden, const uint16_t *__restrict__ w, int R, int V, int d,
    int vtiles, int rblocks, unsigned long long *__restrict__ keys) {
    const int id = blockIdx.x;
    const int local = id / kNumXcd;
    const int vt = (local / rblocks) * kNumXcd + id % kNumXcd;
    const int rb = local % rblocks;
    if (vt >= vtiles) return;                    // whole workgroup, before any barrier
    const int v0 = vt * kTileM, r0 = rb * kTileN;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid & (kWave - 1);

    // Slice loads: instruction i of wave w fills 1 KB block (4w + i) of an
    // operand = rows 16 (4w + i) .. +15; lane p writes row p / 4, position
    // p % 4, which holds chunk (p % 4) ^ ((row >> 2) & 3). Rows past the end
    // of W or hidden read the last row (finite data; results are discarded).
    const char *asrc[kLoads], *bsrc[kLoads];
    {
        const int chunk = (lane & 3) ^ ((lane >> 4) & 3);
        #pragma unroll
        for (int i = 0; i < kLoads; ++i) {
            const int row = (wave * kLoads + i) * 16 + (lane >> 2);
            const int vr = min(v0 + row, V - 1);
            const int hr = min(r0 + row, R - 1);
            asrc[i] = reinterpret_cast<const char *>(w + (size_t)vr * d) + chunk * 16;
            bsrc[i] = reinterpret_cast<const char *>(hidden + (size_t)hr * d) + chunk * 16;
        }
    }
    const int T = d / kBK;

    // Operand fragments of v_mfma_f32_32x32x16_bf16: lane l reads row l % 32
    // of a 32-row block, K elements 8 (l / 32) .. +7 of the 16-deep step, i.e.
    // chunk 2 s + l / 32 of the slice for step s; with the swizzle the chunk's
    // position is (2 s + l / 32) ^ ((l >> 2) & 3) = (base position) ^ 2 s.
    const int wm = wave & 1, wn = wave >> 1;
    const unsigned ring = lds_addr(g_lm_ring);
    const unsigned swz = (unsigned)((((lane >> 5) ^ (lane >> 2)) & 3) << 4);
    const unsigned a_lane = (unsigned)((wm * kWaveM + (lane & 31)) * kSliceRow) + swz;
    const unsigned b_lane = (unsigned)(kOperandBytes + (wn * kWaveN + (lane & 31)) * kSliceRow) + swz;

    f32x16 acc[kFragM][kFragN];
    #pragma unroll
    for (int m = 0; m < kFragM; ++m)
        #pragma unroll
        for (int n = 0; n < kFragN; ++n)
            #pragma unroll
            for (int e = 0; e < 16; ++e) acc[m][n][e] = 0.f;
    u32x4 fa[2][kFragM], fb[2][kFragN];

    auto frag_addr = [&](int stage, int s, unsigned lane_off) {
        return (ring + (unsigned)(stage * kStageBytes) + lane_off) ^ ((unsigned)s << 5);
    };
    // Read q (0..7) of a fragment set: A fragments 0..3, then B fragments 0..3.
    auto read_q = [&](int set, unsigned aa, unsigned ba, int q) {
        if (q < kFragM)
            asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(fa[set][q]) : "v"(aa), "i"(q * 32 * kSliceRow));
        else
            asm volatile("ds_read_b128 %0, %1 offset:%2"
                         : "=v"(fb[set][q - kFragM]) : "v"(ba), "i"((q - kFragM) * 32 * kSliceRow));
    };
    auto ready = [&](int set) {             // after lds_wait_all: the set is in registers
        #pragma unroll
        for (int m = 0; m < kFragM; ++m) tie(fa[set][m]);
        #pragma unroll
        for (int n = 0; n < kFragN; ++n) tie(fb[set][n]);
    };
    auto mfma_q = [&](int set, int q) {
        const int m = q / kFragN, n = q % kFragN;
        acc[m][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8, fa[set][m]), __builtin_bit_cast(bf16x8, fb[set][n]),
            acc[m][n], 0, 0, 0);
    };
    auto issue_load = [&](int t, int i) {     // load i (0 .. 2 kLoads - 1) of slice t
        unsigned char *st = g_lm_ring + (t & (kStages - 1)) * kStageBytes;
        const size_t koff = (size_t)t * kSliceRow;
        if (i < kLoads)
            __builtin_amdgcn_global_load_lds((const GLOBAL_AS void *)(asrc[i] + koff),
                                             (LDS_AS void *)(st + (wave * kLoads + i) * 1024), 16, 0, 0);
        else
            __builtin_amdgcn_global_load_lds((const GLOBAL_AS void *)(bsrc[i - kLoads] + koff),
                                             (LDS_AS void *)(st + kOperandBytes + (wave * kLoads + i - kLoads) * 1024),
                                             16, 0, 0);
    };

    // One K slice j. Step (j, 0) is in fragment set 0 (reads issued earlier).
    // First half: its 16 MFMAs with the reads of step (j, 1) into set 1 between
    // them. Second half: set 1's MFMAs; after the first four, the ring hand-off
    // (slice j + 1 landed everywhere; every wave is done with slice j, whose
    // stage slice j + 4 takes), then the loads of slice j + 4 and the reads of
    // step (j + 1, 0) between the rest. sched_barrier pins the interleaving.
    auto slice = [&](int j, bool more, bool load4, auto wait_next) {
        constexpr int kPre = kSteps / 4;                 // MFMAs before the hand-off
        constexpr int kOps = 2 * kLoads + kReads;        // loads, then reads, after it
        constexpr int kPer = (kOps + kSteps - kPre - 1) / (kSteps - kPre);
        lds_wait_all();
        ready(0);
        {
            const unsigned aa = frag_addr(j & (kStages - 1), 1, a_lane);
            const unsigned ba = frag_addr(j & (kStages - 1), 1, b_lane);
            #pragma unroll
            for (int q = 0; q < kSteps; ++q) {
                mfma_q(0, q);
                if (q < kReads) read_q(1, aa, ba, q);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        lds_wait_all();
        ready(1);
        #pragma unroll
        for (int q = 0; q < kPre; ++q) {
            mfma_q(1, q);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (more) {
            wait_next();
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
        }
        const unsigned aa = frag_addr((j + 1) & (kStages - 1), 0, a_lane);
        const unsigned ba = frag_addr((j + 1) & (kStages - 1), 0, b_lane);
        #pragma unroll
        for (int q = kPre; q < kSteps; ++q) {
            mfma_q(1, q);
            #pragma unroll
            for (int u = 0; u < kPer; ++u) {
                const int op = (q - kPre) * kPer + u;
                if (op < 2 * kLoads) {
                    if (load4) issue_load(j + 4, op);
                } else if (op < kOps) {
                    if (more) read_q(0, aa, ba, op - 2 * kLoads);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // Slices 0..3 in flight; wait for slice 0 (later slices may stay pending).
    #pragma unroll
    for (int t = 0; t < kStages; ++t)
        if (t < T)
            #pragma unroll
            for (int i = 0; i < 2 * kLoads; ++i) issue_load(t, i);
    if (T > 3) wait_vmcnt<6 * kLoads>();
    else if (T > 2) wait_vmcnt<4 * kLoads>();
    else if (T > 1) wait_vmcnt<2 * kLoads>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    {
        const unsigned aa = frag_addr(0, 0, a_lane), ba = frag_addr(0, 0, b_lane);
        #pragma unroll
        for (int q = 0; q < kReads; ++q) read_q(0, aa, ba, q);
    }
    // Steady state: at the hand-off of slice j, slices j + 2 and j + 3 may
    // still be in flight (2 x 2 kLoads loads of this thread).
    int j = 0;
    for (; j + 4 < T; ++j) slice(j, true, true, [] { wait_vmcnt<4 * kLoads>(); });
    for (; j < T; ++j) {
        const int after = T - 2 - j;          // slices issued after j + 1
        slice(j, j + 1 < T, false, [&] {
            if (after >= 2) wait_vmcnt<4 * kLoads>();
            else if (after == 1) wait_vmcnt<2 * kLoads>();
            else wait_vmcnt<0>();
        });
    }

    // Epilogue. acc[m][n][e] of lane l: hidden row 32 n + l % 32 of the wave's
    // block, vocabulary entry 32 m + 8 (e / 4) + 4 (l / 32) + e % 4.
    unsigned long long best[kFragN];
    const int vbase = v0 + wm * kWaveM + 4 * (lane >> 5);
    #pragma unroll
    for (int n = 0; n < kFragN; ++n) {
        unsigned long long b = 0ull;
        #pragma unroll
        for (int m = 0; m < kFragM; ++m)
            #pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int v = vbase + 32 * m + 8 * (e >> 2) + (e & 3);
                const unsigned long long k = pack_key(order_key(acc[m][n][e]), (unsigned)v);
                b = v < V ? umax64(b, k) : b;
            }
        best[n] = halves_max64(b);
    }
    if (wm == 1 && lane < 32) {
        #pragma unroll
        for (int n = 0; n < kFragN; ++n) g_lm_keys[wn][32 * n + lane] = best[n];
    }
    __syncthreads();
    if (wm == 0 && lane < 32) {
        #pragma unroll
        for (int n = 0; n < kFragN; ++n) {
            const int row = r0 + wn * kWaveN + 32 * n + lane;
            if (row < R) atomicMax(keys + row, umax64(best[n], g_lm_keys[wn][32 * n + lane]));
        }
    }
}

}  // namespace

int lm_head_vocab_tiles(int V) { return (int)(((long long)V + kTileM - 1) / kTileM); }

hipError_t launch_lm_head_argmax_accept(const uint16_t *hidden, const uint16_t *w,
                                        const int32_t *draft, const int32_t *parent,
                                        const int32_t *num_nodes, int B, int N, int V, int d,
                                        int32_t *argmax_out, int32_t *accept_len,
                                        int32_t *accept_idx, int32_t *bonus,
                                        unsigned long long *keys, hipStream_t s) {
    if (B == 0) return hipSuccess;
    const int R = B * N;
    hipError_t e = launch_kernel(lm_keys_clear_kernel, dim3((R + 255) / 256), dim3(256), s, keys, R);
    if (e != hipSuccess) return e;
    const int vtiles = lm_head_vocab_tiles(V);
    const int rblocks = (R + kTileN - 1) / kTileN;
    const int groups = (vtiles + kNumXcd - 1) / kNumXcd * kNumXcd * rblocks;
    e = launch_kernel(lm_head_argmax_kernel, dim3(groups), dim3(kLmThreads), s, hidden, w, R, V, d,
                      vtiles, rblocks, keys);
    if (e != hipSuccess) return e;
    return launch_accept(keys, 1, draft, parent, num_nodes, B, N, argmax_out, accept_len,
                         accept_idx, bonus, s);
}

}  // namespace tv
