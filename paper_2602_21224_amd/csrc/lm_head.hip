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
//   * Both operands are K-contiguous (W is [V, d], hidden is [R, d]) and both
//     stream into LDS through global_load_lds_dwordx4, each in its own ring.
//     The weight, which comes from HBM and whose load latency bounds the
//     stream, moves in 64-deep units (each row's 128 bytes = whole cache
//     lines; a 1 KB load covers 8 rows) through a 3-stage ring, two units in
//     flight; the hidden rows, re-read from L2, move in 32-deep slices (16
//     rows x 64 bytes per load) through a 4-stage ring, issued 1.5 units ahead.
//     Together 160 KB: the whole LDS. The 16-byte chunks of each row are
//     XOR-swizzled by the row index so the operand reads (16 rows at one chunk
//     per LDS pass) are free of bank conflicts.
//   * Each 16-deep K step's 8 MFMAs carry, one by one, the next step's 6
//     fragment reads; two ring hand-offs per unit (s_waitcnt vmcnt +
//     s_barrier), a few MFMAs into steps 1 and 3 after this wave's last read of
//     the stages refilled next, are followed by the refill loads.
//   * The four row blocks of one vocabulary tile run together on one XCD and
//     share its L2 copy of the weight tile; each takes the units of every
//     aligned group of four in an order rotated by its row block, so the four
//     ask HBM for different lines at any time (more distinct bytes in flight)
//     and find the others' lines in L2 a few units later.
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
constexpr int kUnitK = 64;                             // K depth of one weight unit
constexpr int kWRow = kUnitK * 2;                      // bytes of one weight row's unit (128)
constexpr int kWUnitBytes = kTileM * kWRow;            // 32 KB
constexpr int kWStages = 3;
constexpr int kHK = 32;                                // K depth of one hidden slice
constexpr int kHRow = kHK * 2;                         // bytes of one hidden row's slice (64)
constexpr int kHSliceBytes = kTileN * kHRow;           // 16 KB
constexpr int kHStages = 4;
constexpr int kWLoads = kWUnitBytes / (kLmThreads * 16);    // 1 KB loads per thread per unit (4)
constexpr int kHLoads = kHSliceBytes / (kLmThreads * 16);   // per slice (2)
constexpr int kWaveM = 128;                            // per-wave block: 2 waves along M
constexpr int kWaveN = kTileN / (kWaves / 2);
constexpr int kFragM = kWaveM / 32, kFragN = kWaveN / 32;
constexpr int kReads = kFragM + kFragN;                // fragment reads per K step
constexpr int kSteps = kFragM * kFragN;                // MFMAs per K step
constexpr int kPre = 2;                                // MFMAs before a hand-off
static_assert(kWLoads * kWaves * 8 == kTileM && kHLoads * kWaves * 16 == kTileN, "load blocks");
static_assert(kWStages * kWUnitBytes + kHStages * kHSliceBytes <= 160 * 1024, "LDS");

__shared__ __attribute__((aligned(1024))) unsigned char g_lm_w[kWStages * kWUnitBytes];
__shared__ __attribute__((aligned(1024))) unsigned char g_lm_h[kHStages * kHSliceBytes];

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

__device__ __forceinline__ void wait_vmcnt_rt(int n) {     // n in {0, 2, 4, 8}
    if (n >= 8) wait_vmcnt<8>();
    else if (n >= 4) wait_vmcnt<4>();
    else if (n >= 2) wait_vmcnt<2>();
    else wait_vmcnt<0>();
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
// d is a multiple of kUnitK.
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
    const int U = d / kUnitK;                    // weight units; hidden slices: 2 U

    // Weight loads: instruction i of wave w fills 1 KB block (4w + i) of a
    // unit = rows 8 (4w + i) .. +7; lane p writes row p / 8, position p % 8,
    // which holds chunk (p % 8) ^ ((row >> 1) & 7). Hidden loads: instruction
    // i fills block (2w + i) of a slice = rows 16 (2w + i) .. +15; lane p
    // writes row p / 4, position p % 4 = chunk (p % 4) ^ ((row >> 2) & 3).
    // Rows past the end of W or hidden read the last row (finite data; the
    // results are discarded).
    const char *wsrc[kWLoads], *hsrc[kHLoads];
    {
        #pragma unroll
        for (int i = 0; i < kWLoads; ++i) {
            const int row = (wave * kWLoads + i) * 8 + (lane >> 3);
            const int chunk = (lane & 7) ^ ((row >> 1) & 7);
            wsrc[i] = reinterpret_cast<const char *>(w + (size_t)min(v0 + row, V - 1) * d) + chunk * 16;
        }
        #pragma unroll
        for (int i = 0; i < kHLoads; ++i) {
            const int row = (wave * kHLoads + i) * 16 + (lane >> 2);
            const int chunk = (lane & 3) ^ ((row >> 2) & 3);
            hsrc[i] = reinterpret_cast<const char *>(hidden + (size_t)min(r0 + row, R - 1) * d) + chunk * 16;
        }
    }
    // Unit order: inside every complete aligned group of four, rotated by the
    // row block (a permutation of 0 .. U - 1).
    const int U4 = U & ~3;
    auto unit_of = [&](int u) { return u < U4 ? (u & ~3) | ((u + rb) & 3) : u; };
    // Load i of a weight unit / hidden slice: LDS stage offset, K byte offset.
    auto issue_w = [&](unsigned stage_off, size_t koff, int i) {
        __builtin_amdgcn_global_load_lds((const GLOBAL_AS void *)(wsrc[i] + koff),
                                         (LDS_AS void *)(g_lm_w + stage_off + (wave * kWLoads + i) * 1024),
                                         16, 0, 0);
    };
    auto issue_h = [&](unsigned stage_off, size_t koff, int i) {
        __builtin_amdgcn_global_load_lds((const GLOBAL_AS void *)(hsrc[i] + koff),
                                         (LDS_AS void *)(g_lm_h + stage_off + (wave * kHLoads + i) * 1024),
                                         16, 0, 0);
    };

    // Operand fragments of v_mfma_f32_32x32x16_bf16: lane l reads row l % 32
    // of a 32-row block, K elements 8 (l / 32) .. +7 of the 16-deep step.
    // Step s (0..3) of a unit is weight chunk 2 s + l / 32, whose position is
    // (l / 32) ^ ((row >> 1) & 7) ^ 2 s, and hidden slice s / 2, chunk
    // 2 (s % 2) + l / 32 at position (l / 32) ^ ((row >> 2) & 3) ^ 2 (s % 2).
    const int wm = wave & 1, wn = wave >> 1;
    const unsigned wring = lds_addr(g_lm_w), hring = lds_addr(g_lm_h);
    const unsigned a_lane = wring + (unsigned)((wm * kWaveM + (lane & 31)) * kWRow) +
                            (unsigned)((((lane >> 5) ^ (lane >> 1)) & 7) << 4);
    const unsigned b_lane = hring + (unsigned)((wn * kWaveN + (lane & 31)) * kHRow) +
                            (unsigned)((((lane >> 5) ^ (lane >> 2)) & 3) << 4);

    f32x16 acc[kFragM][kFragN];
    #pragma unroll
    for (int m = 0; m < kFragM; ++m)
        #pragma unroll
        for (int n = 0; n < kFragN; ++n)
            #pragma unroll
            for (int e = 0; e < 16; ++e) acc[m][n][e] = 0.f;
    u32x4 fa[2][kFragM], fb[2][kFragN];

    // Read q (0..5) of a fragment set: A fragments 0..3, then B fragments 0..1.
    auto read_q = [&](int set, unsigned aa, unsigned ba, int q) {
        if (q < kFragM)
            asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(fa[set][q]) : "v"(aa), "i"(q * 32 * kWRow));
        else
            asm volatile("ds_read_b128 %0, %1 offset:%2"
                         : "=v"(fb[set][q - kFragM]) : "v"(ba), "i"((q - kFragM) * 32 * kHRow));
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

    // Issue order, the same in the prologue and the steady state: hand-off A
    // of unit u (in step 1) issues hidden slice 2u + 4; hand-off B (in step 3)
    // issues weight unit u + 3, then hidden slice 2u + 5. Stages: weight unit
    // x in x % 3, hidden slice x in x % 4. The prologue plays hand-offs
    // B(-3), A(-2), B(-2), A(-1), B(-1).
    {
        const size_t k0 = (size_t)unit_of(0) * kWRow, k1 = (size_t)unit_of(1) * kWRow;
        #pragma unroll
        for (int i = 0; i < kWLoads; ++i) issue_w(0, k0, i);                          // W0
        #pragma unroll
        for (int i = 0; i < kHLoads; ++i) issue_h(0, k0, i);                          // H0
        if (U >= 2)
            #pragma unroll
            for (int i = 0; i < kWLoads; ++i) issue_w(kWUnitBytes, k1, i);            // W1
        #pragma unroll
        for (int i = 0; i < kHLoads; ++i) issue_h(kHSliceBytes, k0 + kHRow, i);       // H1
        if (U >= 2)
            #pragma unroll
            for (int i = 0; i < kHLoads; ++i) issue_h(2 * kHSliceBytes, k1, i);       // H2
        if (U >= 3) {
            const size_t k2 = (size_t)unit_of(2) * kWRow;
            #pragma unroll
            for (int i = 0; i < kWLoads; ++i) issue_w(2 * kWUnitBytes, k2, i);        // W2
        }
        if (U >= 2)
            #pragma unroll
            for (int i = 0; i < kHLoads; ++i) issue_h(3 * kHSliceBytes, k1 + kHRow, i);   // H3
        // Unit 0 needs W0 and H0; what came after may stay in flight.
        if (U >= 3) wait_vmcnt<kHLoads + kWLoads + 2 * kHLoads + kWLoads>();
        else if (U >= 2) wait_vmcnt<kHLoads + kWLoads + 2 * kHLoads>();
        else wait_vmcnt<kHLoads>();
    }
    __builtin_amdgcn_s_barrier();
    #pragma unroll
    for (int q = 0; q < kReads; ++q) read_q(0, a_lane, b_lane, q);

    // One unit u (4 steps of 16). Step s's fragments are in set s & 1. Steps 0
    // and 2: 8 MFMAs with the next step's 6 reads between them. Steps 1 and 3:
    // kPre MFMAs, the hand-off (the data of the next reads landed everywhere;
    // every wave is done with the stages refilled now), then the remaining
    // MFMAs carrying the hand-off's loads and then the next step's reads.
    // sched_barrier pins the interleaving. kSteady: u + 3 < U, so every load
    // of the hand-offs exists and the waits are constant.
    int wst = 0;                                      // weight stage of unit u
    auto unit = [&](int u, auto steady_c) {
        constexpr bool kSteady = decltype(steady_c)::value;
        const unsigned wcur = (unsigned)wst * kWUnitBytes;
        const unsigned wnxt = (unsigned)(wst == kWStages - 1 ? 0 : wst + 1) * kWUnitBytes;
        const unsigned hcur = (unsigned)(u & 1) * 2 * kHSliceBytes;     // stage of slice 2u
        const unsigned a0 = a_lane + wcur, a1 = a_lane + wnxt;
        const unsigned b0 = b_lane + hcur, b1 = b_lane + (hcur ^ 2 * kHSliceBytes);
        const size_t kw = (size_t)unit_of(u + 3) * kWRow;              // weight unit u + 3
        const size_t kh = (size_t)unit_of(u + 2) * kWRow;              // hidden slices 2u + 4, 2u + 5
        const bool has_w = kSteady || u + 3 < U;
        const bool has_h = kSteady || u + 2 < U;
        const bool has_next = kSteady || u + 1 < U;

        auto step = [&](auto sc) {
            constexpr int s = decltype(sc)::value;
            constexpr int set = s & 1;
            const unsigned aa = s == 3 ? a1 : a0 ^ ((unsigned)(s + 1) << 5);
            const unsigned ba = s == 3 ? b1
                                       : (b0 + (unsigned)(((s + 1) >> 1) * kHSliceBytes)) ^
                                             ((unsigned)((s + 1) & 1) << 5);
            lds_wait_all();
            ready(set);
            if constexpr (s == 0 || s == 2) {
                #pragma unroll
                for (int q = 0; q < kSteps; ++q) {
                    mfma_q(set, q);
                    if (q < kReads) read_q(set ^ 1, aa, ba, q);
                    __builtin_amdgcn_sched_barrier(0);
                }
            } else {
                constexpr int kLoadsHere = s == 1 ? kHLoads : kWLoads + kHLoads;
                constexpr int kOps = kLoadsHere + kReads;
                constexpr int kPer = (kOps + kSteps - kPre - 1) / (kSteps - kPre);
                const bool next = s == 1 || has_next;
                #pragma unroll
                for (int q = 0; q < kPre; ++q) {
                    mfma_q(set, q);
                    __builtin_amdgcn_sched_barrier(0);
                }
                if (next) {
                    // loads issued after the newest one the next reads need
                    if constexpr (kSteady) {
                        wait_vmcnt<2 * kWLoads>();
                    } else if constexpr (s == 1) {   // hidden slice 2u + 1 (from B(u - 2))
                        wait_vmcnt_rt((u + 1 < U ? 4 : 0) + (u + 2 < U ? 4 : 0));
                    } else {                         // unit u + 1 (B(u - 2)), slice 2u + 2 (A(u - 1))
                        wait_vmcnt_rt((u + 2 < U ? 6 : 0) + (u + 1 < U ? 2 : 0));
                    }
                    __builtin_amdgcn_s_barrier();
                    __builtin_amdgcn_sched_barrier(0);
                }
                #pragma unroll
                for (int q = kPre; q < kSteps; ++q) {
                    mfma_q(set, q);
                    #pragma unroll
                    for (int x = 0; x < kPer; ++x) {
                        const int op = (q - kPre) * kPer + x;
                        if (op < kLoadsHere) {
                            if (s == 1) {
                                if (has_h) issue_h(hcur, kh, op);                       // slice 2u + 4
                            } else if (op < kWLoads) {
                                if (has_w) issue_w(wcur, kw, op);                       // unit u + 3
                            } else if (has_h) {
                                issue_h(hcur + kHSliceBytes, kh + kHRow, op - kWLoads); // slice 2u + 5
                            }
                        } else if (op < kOps) {
                            if (next) read_q(set ^ 1, aa, ba, op - kLoadsHere);
                        }
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        };
        step(std::integral_constant<int, 0>());
        step(std::integral_constant<int, 1>());
        step(std::integral_constant<int, 2>());
        step(std::integral_constant<int, 3>());
        wst = wst == kWStages - 1 ? 0 : wst + 1;
    };
    int u = 0;
    for (; u + 3 < U; ++u) unit(u, std::true_type());
    for (; u < U; ++u) unit(u, std::false_type());

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
    // The keys of the two M-waves meet in LDS (the hidden ring, free once
    // every wave is past its last fragment read).
    unsigned long long *kx = reinterpret_cast<unsigned long long *>(g_lm_h);
    __syncthreads();
    if (wm == 1 && lane < 32) {
        #pragma unroll
        for (int n = 0; n < kFragN; ++n) kx[wn * kWaveN + 32 * n + lane] = best[n];
    }
    __syncthreads();
    if (wm == 0 && lane < 32) {
        #pragma unroll
        for (int n = 0; n < kFragN; ++n) {
            const int row = r0 + wn * kWaveN + 32 * n + lane;
            if (row < R) atomicMax(keys + row, umax64(best[n], kx[wn * kWaveN + 32 * n + lane]));
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
