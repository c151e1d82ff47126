// C-ABI entry points of libtreeverify: argument checks, launch shapes and
// workspace carving. Every check runs on the host before any launch, so an
// error return means nothing was enqueued.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <atomic>

#define TREEVERIFY_BUILD 1
#include "treeverify.h"
#include "tv_internal.h"

namespace {

constexpr int kMaxDevices = 64;
constexpr int kWgPerCu = 1;          // the attention kernel's LDS ring allows one workgroup per CU
constexpr int kMinShareTiles = 2;    // smallest per-workgroup share (measured: 8 -> 2 is -26 % at 8B bs1)
constexpr int kSetupTiles = 3;       // measured cost of starting a unit piece, in 64-key tiles
constexpr int kArgmaxMinWorkgroups = 2048;
constexpr int kArgmaxMinSegment = 4096;

int g_cu_count[kMaxDevices];         // 0 = not yet queried
int g_is_gfx950[kMaxDevices];        // 0 = not yet queried, 1 = yes, -1 = no

// Scratch of tree_argmax_accept_noalloc: one copy per GPU, held until the
// process ends. Host code never names it directly (its host-side name is a
// stand-in, not a device address); it uses the per-device address that
// hipGetSymbolAddress returns, looked up once per device on the first call.
static __device__ __align__(256) unsigned char scratch[TV_NOALLOC_SCRATCH_BYTES];
std::atomic<void *> g_scratch_ptr[kMaxDevices];

// Device address of the current device's scratch, or nullptr if the lookup fails.
void *scratch_ptr() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    void *ptr = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (ptr == nullptr) {
        // Two threads may race here; both store the same address.
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr)
            return nullptr;
        g_scratch_ptr[dev].store(ptr, std::memory_order_release);
    }
    return ptr;
}

bool device_ok() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return false;
    if (g_is_gfx950[dev] == 0) {
        hipDeviceProp_t prop;
        const bool ok = hipGetDeviceProperties(&prop, dev) == hipSuccess &&
                        strncmp(prop.gcnArchName, "gfx950", 6) == 0;
        g_is_gfx950[dev] = ok ? 1 : -1;
    }
    return g_is_gfx950[dev] == 1;
}

int cu_count() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
    if (g_cu_count[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        g_cu_count[dev] = n;
    }
    return g_cu_count[dev];
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }
size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct AttnShape {
    int G, rows, waves, rows_per_block, row_blocks, tree_tiles_all;
};

AttnShape attn_shape(int N, int Hq, int Hkv) {
    AttnShape s;
    s.G = Hq / Hkv;
    s.rows = N * s.G;
    // Four waves at least: a workgroup of fewer waves leaves a unit's tile
    // loads to one or two waves (and the one-wave kernel spills), which
    // measured 11x (one wave) and 1.2x (two waves) slower on 12-row units
    // than four waves with the extra rows idle.
    const int need = (s.rows + tv::kRowsPerWave - 1) / tv::kRowsPerWave;
    s.waves = need > 4 ? 8 : 4;
    s.rows_per_block = s.waves * tv::kRowsPerWave;
    s.row_blocks = (s.rows + s.rows_per_block - 1) / s.rows_per_block;
    s.tree_tiles_all = 0;
    for (int rb = 0; rb < s.row_blocks; ++rb) {
        const int last_row = (rb + 1) * s.rows_per_block < s.rows ? (rb + 1) * s.rows_per_block - 1
                                                                  : s.rows - 1;
        const int jmax = last_row / s.G + 1;
        s.tree_tiles_all += (jmax + tv::kKeyTile - 1) / tv::kKeyTile;
    }
    return s;
}

struct AttnWorkspace {
    size_t o_bytes, ml_bytes, desc_bytes, total;
};

AttnWorkspace attn_workspace(const AttnShape &s, int D, int max_wg) {
    AttnWorkspace w;
    w.o_bytes = round_up((size_t)max_wg * 2 * s.rows_per_block * D * sizeof(uint16_t), 256);
    w.ml_bytes = round_up((size_t)max_wg * 2 * s.rows_per_block * 2 * sizeof(float), 256);
    w.desc_bytes = round_up((size_t)max_wg * 4 * sizeof(int32_t), 256);
    w.total = w.o_bytes + w.ml_bytes + w.desc_bytes;
    return w;
}

bool attn_shape_ok(int B, int N, int Hq, int Hkv, int D) {
    if (B < 0 || B > tv::kMaxBatchAttn) return false;
    if (N < 1 || N > tv::kMaxNodes) return false;
    if (D != 64 && D != 128) return false;
    if (Hq < 1 || Hkv < 1 || Hq % Hkv != 0) return false;
    if ((long)(Hq / Hkv) * N > 2048) return false;
    // 256 key rows of all KV heads (a page, or the tree's rows) stay below 4 GiB,
    // so in-kernel row offsets fit 32 bits
    if ((long)Hkv * D * 2 * 256 >= (1l << 32)) return false;
    return true;
}

void argmax_plan(int B, int N, int V, int *segs, int *seg_len) {
    const long rows = (long)B * N;
    long s = rows > 0 ? (kArgmaxMinWorkgroups + rows - 1) / rows : 1;
    const long max_s = ((long)V + kArgmaxMinSegment - 1) / kArgmaxMinSegment;
    if (s > max_s) s = max_s;
    if (s < 1) s = 1;
    if (s > 65535) s = 65535;
    long len = ((long)V + s - 1) / s;
    len = (len + 3) / 4 * 4;
    s = ((long)V + len - 1) / len;
    *segs = (int)s;
    *seg_len = (int)len;
}

}  // namespace

extern "C" {

int tv_abi_version(void) { return TV_ABI_VERSION; }

const char *tv_status_string(int status) {
    switch (status) {
        case TV_OK: return "ok";
        case TV_ERR_NULL: return "a required pointer is NULL";
        case TV_ERR_SHAPE: return "a size or count is outside the supported range";
        case TV_ERR_ALIGN: return "a tensor pointer is not 16-byte aligned";
        case TV_ERR_WORKSPACE: return "workspace missing or smaller than required";
        case TV_ERR_HIP: return "a HIP runtime call or kernel launch failed";
        case TV_ERR_DEVICE: return "the current device is not gfx950";
        case TV_ERR_SCRATCH:
            return "the call needs more scratch than the library's static buffer holds "
                   "(TV_NOALLOC_SCRATCH_BYTES)";
        default: return "unknown status";
    }
}

size_t tv_attention_workspace_size(int B, int N, int Hq, int Hkv, int D) {
    if (!attn_shape_ok(B, N, Hq, Hkv, D)) return 0;
    const AttnShape s = attn_shape(N, Hq, Hkv);
    return attn_workspace(s, D, cu_count() * kWgPerCu).total;
}

int tree_verify_attention(const uint16_t *q, const uint16_t *k_tree, const uint16_t *v_tree,
                          const uint16_t *k_cache, const uint16_t *v_cache,
                          const int32_t *page_table, const int32_t *kv_len, const int32_t *parent,
                          const int32_t *num_nodes, int B, int N, int Hq, int Hkv, int D, int P,
                          int max_pages, int num_pages, int max_kv_len, float scale, uint16_t *out,
                          float *lse,
                          void *workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!attn_shape_ok(B, N, Hq, Hkv, D)) return TV_ERR_SHAPE;
    if (!pow2(P) || P > 256 || max_pages < 1 || num_pages < 1 || max_kv_len < 0)
        return TV_ERR_SHAPE;
    if (B == 0) return TV_OK;
    if (!q || !k_tree || !v_tree || !k_cache || !v_cache || !page_table || !kv_len || !parent ||
        !out || !workspace)
        return TV_ERR_NULL;
    if (!aligned16(q) || !aligned16(k_tree) || !aligned16(v_tree) || !aligned16(k_cache) ||
        !aligned16(v_cache) || !aligned16(out) || !aligned16(workspace))
        return TV_ERR_ALIGN;
    if (!device_ok()) return TV_ERR_DEVICE;

    const AttnShape s = attn_shape(N, Hq, Hkv);
    const int max_wg = cu_count() * kWgPerCu;
    const AttnWorkspace ws = attn_workspace(s, D, max_wg);
    if (workspace_bytes < ws.total) return TV_ERR_WORKSPACE;

    // the (virtual) tile count of the whole launch must fit in int32 for any kv_len
    const long max_len = (long)max_pages * P;
    const long worst = (long)B * Hkv *
                       ((long)s.row_blocks * ((max_len + tv::kKeyTile - 1) / tv::kKeyTile + kSetupTiles) +
                        s.tree_tiles_all);
    if (worst >= (1l << 30)) return TV_ERR_SHAPE;

    const long hint_len = max_kv_len < max_len ? max_kv_len : max_len;
    const long est = (long)B * Hkv *
                     ((long)s.row_blocks * ((hint_len + tv::kKeyTile - 1) / tv::kKeyTile + kSetupTiles) +
                      s.tree_tiles_all);
    long num_wg = est / kMinShareTiles;
    if (num_wg < 1) num_wg = 1;
    if (num_wg > max_wg) num_wg = max_wg;

    tv::AttnParams p;
    p.q = q; p.k_tree = k_tree; p.v_tree = v_tree; p.k_cache = k_cache; p.v_cache = v_cache;
    p.page_table = page_table; p.kv_len = kv_len; p.parent = parent; p.num_nodes = num_nodes;
    p.out = out; p.lse = lse;
    char *base = static_cast<char *>(workspace);
    p.ws_o = reinterpret_cast<uint16_t *>(base);
    p.ws_ml = reinterpret_cast<float *>(base + ws.o_bytes);
    p.ws_desc = reinterpret_cast<int32_t *>(base + ws.o_bytes + ws.ml_bytes);
    p.B = B; p.N = N; p.Hq = Hq; p.Hkv = Hkv; p.G = s.G;
    p.P = P; p.p_shift = __builtin_ctz((unsigned)P);
    p.max_pages = max_pages; p.num_pages = num_pages;
    p.rows_per_block = s.rows_per_block;
    p.setup_tiles = kSetupTiles;
    p.small_pages = P < 1024 / (2 * D) ? 1 : 0;
    p.narrow = s.rows <= 16 ? 1 : 0;
    p.num_wg = (int)num_wg;
    const float sc = scale > 0.f ? scale : 1.0f / sqrtf((float)D);
    p.scale = sc;
    p.scale_log2 = sc * 1.4426950408889634f;

    return tv::launch_tree_attention(p, D, s.waves, stream) == hipSuccess ? TV_OK : TV_ERR_HIP;
}

size_t tv_argmax_workspace_size(int B, int N, int V) {
    if (B < 0 || B > 65535 || N < 1 || N > tv::kMaxNodes || V < 1) return 0;
    int segs = 1, seg_len = 4;
    argmax_plan(B, N, V, &segs, &seg_len);
    return round_up((size_t)B * N * segs * sizeof(unsigned long long), 256) + 256;
}

}  // extern "C"

namespace {

// Argument checks and launches shared by tree_argmax_accept and its no-alloc
// variant; `ws` is the per-(row, segment) key buffer (every slot the accept
// kernel reads is written earlier in the same call).
int argmax_accept_checked(const float *logits, const int32_t *draft_tokens, const int32_t *parent,
                          const int32_t *num_nodes, int B, int N, int V, int32_t *argmax_out,
                          int32_t *accept_len, int32_t *accept_idx, int32_t *bonus_token,
                          void *ws, hipStream_t stream) {
    int segs = 1, seg_len = 4;
    argmax_plan(B, N, V, &segs, &seg_len);
    const hipError_t e = tv::launch_argmax_accept(
        logits, draft_tokens, parent, num_nodes, B, N, V, segs, seg_len, argmax_out, accept_len,
        accept_idx, bonus_token, static_cast<unsigned long long *>(ws), stream);
    return e == hipSuccess ? TV_OK : TV_ERR_HIP;
}

bool argmax_args_ok(int B, int N, int V) {
    return B >= 0 && B <= 65535 && N >= 1 && N <= tv::kMaxNodes && V >= 1;
}

bool argmax_ptrs_ok(const float *logits, const int32_t *draft_tokens, const int32_t *parent,
                    int32_t *argmax_out, int32_t *accept_len, int32_t *accept_idx,
                    int32_t *bonus_token) {
    return logits && draft_tokens && parent && argmax_out && accept_len && accept_idx &&
           bonus_token;
}

}  // namespace

extern "C" {

int tree_argmax_accept(const float *logits, const int32_t *draft_tokens, const int32_t *parent,
                       const int32_t *num_nodes, int B, int N, int V, int32_t *argmax_out,
                       int32_t *accept_len,
                       int32_t *accept_idx, int32_t *bonus_token, void *workspace,
                       size_t workspace_bytes, hipStream_t stream) {
    if (!argmax_args_ok(B, N, V)) return TV_ERR_SHAPE;
    if (B == 0) return TV_OK;
    if (!argmax_ptrs_ok(logits, draft_tokens, parent, argmax_out, accept_len, accept_idx,
                        bonus_token) || !workspace)
        return TV_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(logits) & 3u) || (reinterpret_cast<uintptr_t>(workspace) & 7u))
        return TV_ERR_ALIGN;
    if (workspace_bytes < tv_argmax_workspace_size(B, N, V)) return TV_ERR_WORKSPACE;
    if (!device_ok()) return TV_ERR_DEVICE;
    return argmax_accept_checked(logits, draft_tokens, parent, num_nodes, B, N, V, argmax_out,
                                 accept_len, accept_idx, bonus_token, workspace, stream);
}

int tree_argmax_accept_noalloc(const float *logits, const int32_t *draft_tokens,
                               const int32_t *parent, const int32_t *num_nodes, int B, int N,
                               int V, int32_t *argmax_out, int32_t *accept_len,
                               int32_t *accept_idx, int32_t *bonus_token, hipStream_t stream) {
    if (!argmax_args_ok(B, N, V)) return TV_ERR_SHAPE;
    if (B == 0) return TV_OK;
    if (!argmax_ptrs_ok(logits, draft_tokens, parent, argmax_out, accept_len, accept_idx,
                        bonus_token))
        return TV_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(logits) & 3u) return TV_ERR_ALIGN;
    if (tv_argmax_workspace_size(B, N, V) > (size_t)TV_NOALLOC_SCRATCH_BYTES)
        return TV_ERR_SCRATCH;
    if (!device_ok()) return TV_ERR_DEVICE;
    void *ws = scratch_ptr();
    if (ws == nullptr) return TV_ERR_HIP;
    return argmax_accept_checked(logits, draft_tokens, parent, num_nodes, B, N, V, argmax_out,
                                 accept_len, accept_idx, bonus_token, ws, stream);
}

int kv_compact_accepted(const uint16_t *k_tree, const uint16_t *v_tree, uint16_t *k_cache,
                        uint16_t *v_cache, const int32_t *page_table, const int32_t *kv_len,
                        const int32_t *accept_idx, const int32_t *accept_len, int B, int N,
                        int Hkv, int D, int P, int max_pages, int num_pages, hipStream_t stream) {
    if (B < 0 || B > 65535 || N < 1 || N > tv::kMaxNodes || Hkv < 1 || D < 1 ||
        ((long)Hkv * D) % 8 != 0 || !pow2(P) || P > 256 || max_pages < 1 || num_pages < 1)
        return TV_ERR_SHAPE;
    if (B == 0) return TV_OK;
    if (!k_tree || !v_tree || !k_cache || !v_cache || !page_table || !kv_len || !accept_idx ||
        !accept_len)
        return TV_ERR_NULL;
    if (!aligned16(k_tree) || !aligned16(v_tree) || !aligned16(k_cache) || !aligned16(v_cache))
        return TV_ERR_ALIGN;
    if (!device_ok()) return TV_ERR_DEVICE;
    const hipError_t e = tv::launch_kv_compact(k_tree, v_tree, k_cache, v_cache, page_table,
                                               kv_len, accept_idx, accept_len, B, N, Hkv, D, P,
                                               max_pages, num_pages, stream);
    return e == hipSuccess ? TV_OK : TV_ERR_HIP;
}

int tv_validate_inputs(const int32_t *page_table, const int32_t *kv_len, const int32_t *parent,
                       const int32_t *num_nodes, int B, int N, int P, int max_pages,
                       int num_pages, int32_t *status_word, hipStream_t stream) {
    if (B < 0 || N < 1 || N > tv::kMaxNodes || !pow2(P) || max_pages < 1 || num_pages < 1)
        return TV_ERR_SHAPE;
    if (!status_word || (B > 0 && (!page_table || !kv_len || !parent))) return TV_ERR_NULL;
    if (!device_ok()) return TV_ERR_DEVICE;
    const hipError_t e = tv::launch_validate(page_table, kv_len, parent, num_nodes, B, N, P,
                                             max_pages, num_pages, status_word, stream);
    return e == hipSuccess ? TV_OK : TV_ERR_HIP;
}

static bool tree_build_shape_ok(int B, int S, int V, int H, int k) {
    return B >= 0 && B <= 65535 && S >= 1 && S <= tv::kTbMaxSteps && V >= 1 && H >= 0 &&
           H <= V && k >= 1 && k <= tv::kTbMaxK && k <= V;
}

size_t tv_tree_build_workspace_size(int B, int S, int V, int H, int k) {
    if (!tree_build_shape_ok(B, S, V, H, k)) return 0;
    const tv::TreeBuildPlan pl = tv::tree_build_plan(B, S, V, H, k);
    const size_t nn = (size_t)B * pl.max_nodes;
    return round_up(pl.rows_bytes, 256) + round_up(pl.parts_bytes, 256) +
           round_up(pl.hot_logits_bytes, 256) +
           2 * round_up(nn * sizeof(int32_t), 256) + round_up(nn * sizeof(double), 256) +
           round_up(pl.frontier_bytes, 256) + 256;
}

int tree_build(const float *logits, const int32_t *root_token, const uint16_t *token_info,
               const int32_t *hot_vocab, const int32_t *hot_index, int B, int S, int V, int H,
               int k, int budget, int32_t *parent, int32_t *token, float *joint,
               int32_t *num_nodes, void *workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!tree_build_shape_ok(B, S, V, H, k) || budget < 1 || budget > tv::kMaxNodes)
        return TV_ERR_SHAPE;
    if (B == 0) return TV_OK;
    if (!logits || !root_token || !parent || !token || !joint || !num_nodes || !workspace ||
        (H > 0 && (!token_info || !hot_vocab || !hot_index)))
        return TV_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(logits) & 3u) || (reinterpret_cast<uintptr_t>(workspace) & 7u))
        return TV_ERR_ALIGN;
    if (workspace_bytes < tv_tree_build_workspace_size(B, S, V, H, k)) return TV_ERR_WORKSPACE;
    if (!device_ok()) return TV_ERR_DEVICE;
    const hipError_t e = tv::launch_tree_build(logits, root_token, token_info, hot_vocab,
                                               hot_index, nullptr, 0, B, S, V, H, k, budget,
                                               parent, token, joint, num_nodes, workspace,
                                               stream);
    return e == hipSuccess ? TV_OK : TV_ERR_HIP;
}

int tree_resample(const float *logits, const int32_t *bonus_token, const int32_t *accept_len,
                  const uint16_t *token_info, const int32_t *hot_vocab, const int32_t *hot_index,
                  int B, int S, int V, int H, int k, int r, int budget, int32_t *parent,
                  int32_t *token, float *joint, int32_t *num_nodes, void *workspace,
                  size_t workspace_bytes, hipStream_t stream) {
    if (!tree_build_shape_ok(B, S, V, H, k) || budget < 1 || budget > tv::kMaxNodes || r < 0)
        return TV_ERR_SHAPE;
    if (B == 0) return TV_OK;
    if (!logits || !bonus_token || !accept_len || !parent || !token || !joint || !num_nodes ||
        !workspace || (H > 0 && (!token_info || !hot_vocab || !hot_index)))
        return TV_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(logits) & 3u) || (reinterpret_cast<uintptr_t>(workspace) & 7u))
        return TV_ERR_ALIGN;
    if (workspace_bytes < tv_tree_build_workspace_size(B, S, V, H, k)) return TV_ERR_WORKSPACE;
    if (!device_ok()) return TV_ERR_DEVICE;
    const hipError_t e = tv::launch_tree_build(logits, bonus_token, token_info, hot_vocab,
                                               hot_index, accept_len, r, B, S, V, H, k, budget,
                                               parent, token, joint, num_nodes, workspace,
                                               stream);
    return e == hipSuccess ? TV_OK : TV_ERR_HIP;
}

static bool lm_head_shape_ok(int B, int N, int V, int d) {
    // V: vocabulary ids of a tile's rows (v0 + 0..255) must fit an int
    if (B < 0 || B > 65535 || N < 1 || N > tv::kMaxNodes || V < 1 || V > 0x7FFFFFFF - 256 ||
        d < 64 || d % 64 != 0)
        return false;
    const long long rblocks = ((long long)B * N + 255) / 256;
    const long long groups = ((long long)tv::lm_head_vocab_tiles(V) + 7) / 8 * 8 * rblocks;
    return groups <= 0x7FFFFFFFll;
}

size_t tv_lm_head_workspace_size(int B, int N, int V, int d) {
    if (!lm_head_shape_ok(B, N, V, d)) return 0;
    return round_up((size_t)B * N * sizeof(unsigned long long), 256) + 256;
}

int tree_lm_head_argmax_accept(const uint16_t *hidden, const uint16_t *w_head,
                               const int32_t *draft_tokens, const int32_t *parent,
                               const int32_t *num_nodes, int B, int N, int V, int d,
                               int32_t *argmax_out, int32_t *accept_len, int32_t *accept_idx,
                               int32_t *bonus_token, void *workspace, size_t workspace_bytes,
                               hipStream_t stream) {
    if (!lm_head_shape_ok(B, N, V, d)) return TV_ERR_SHAPE;
    if (B == 0) return TV_OK;
    if (!hidden || !w_head || !draft_tokens || !parent || !argmax_out || !accept_len ||
        !accept_idx || !bonus_token || !workspace)
        return TV_ERR_NULL;
    if (!aligned16(hidden) || !aligned16(w_head) || (reinterpret_cast<uintptr_t>(workspace) & 7u))
        return TV_ERR_ALIGN;
    if (workspace_bytes < tv_lm_head_workspace_size(B, N, V, d)) return TV_ERR_WORKSPACE;
    if (!device_ok()) return TV_ERR_DEVICE;
    const hipError_t e = tv::launch_lm_head_argmax_accept(
        hidden, w_head, draft_tokens, parent, num_nodes, B, N, V, d, argmax_out, accept_len,
        accept_idx, bonus_token, static_cast<unsigned long long *>(workspace), stream);
    return e == hipSuccess ? TV_OK : TV_ERR_HIP;
}

}  // extern "C"
