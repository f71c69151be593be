// Internal interface between the host-side validation/planning code
// (ws_api.cpp, no HIP headers) and the gfx950 kernels (ws_kernels.hip for
// attention, merge and append; ws_bwd.hip for the gradients).
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace ws {

enum { MODE_PREFILL = 0, MODE_STEP = 1 };

constexpr int MAX_SPLITS = 32;   // KV splits of one step at most
// MI355X: 8 XCDs; work-groups are dispatched to them round-robin, and the
// attention kernel gives XCD x the contiguous work items
// [x * per_xcd, (x + 1) * per_xcd)
constexpr int NUM_XCD = 8;

// Division by a divisor d (1 <= d < 2^31) fixed for a launch, exact for
// dividends n < 2^31: with l = ceil(log2 d), mul = ceil(2^(31+l) / d) and
// shift = 31 + l, n / d = (n * mul) >> shift (the round-up method of
// Granlund and Montgomery, "Division by invariant integers using
// multiplication", 1994).  mul < 2^32, and the error term n * (mul * d -
// 2^(31+l)) / 2^(31+l) stays below 1 because n < 2^31 and mul * d -
// 2^(31+l) < d <= 2^l.
struct FastDiv {
    uint32_t mul;
    uint32_t shift;
};

inline FastDiv fastdiv_make(uint32_t d) {
    uint32_t l = 0;
    while (l < 31 && (1u << l) < d) ++l;
    const uint64_t num = (uint64_t)1 << (31 + l);
    FastDiv f;
    f.mul = (uint32_t)((num + d - 1) / d);
    f.shift = 31 + l;
    return f;
}

// Everything one attention launch needs.  Element strides; bf16 data is
// carried as uint16_t bit patterns.
struct AttnArgs {
    // queries [B][Lq][Hq][D]
    const uint16_t *q;
    int64_t q_sb, q_st, q_sh;
    // contiguous keys/values: the prefill's K/V, or the step's own new block
    const uint16_t *kc, *vc;
    int64_t kc_sb, kc_st, kc_sh;
    int64_t vc_sb, vc_st, vc_sh;
    // paged pool [pages][Hkv][64][D] and its table [B][max_pages]
    uint16_t *kpool, *vpool;
    const int32_t *page_table;
    int32_t max_pages;
    // step: cache length of each stream [B]; prefill: block offsets [B][nb+1]
    const int32_t *cache_lens;
    const int32_t *offsets;
    int32_t nb;
    // token-causal segments (has_text): step [B] starts within the new
    // block; prefill [B][nb] absolute starts.  Token i of a block sees the
    // keys j < max(start, i + 1) (prefill positions; step: n_pool + that).
    const int32_t *text_starts;
    int32_t has_text;
    // step: tokens of each stream's new block [B] (has_new_lens; else Lq).
    // New token t sees n_pool + min(new_len_b, max(start, t + 1)) keys;
    // tokens past new_len_b are padding: never keys, never committed, and
    // tiles (and combine rows) of padding only are skipped.
    const int32_t *new_lens;
    int32_t has_new_lens;
    // output [B][Lq][Hq][D] (bf16 or f32) and lse [B][Hq][Lq] (nullable)
    void *out;
    int64_t o_sb, o_st, o_sh;
    int32_t out_f32;
    float *lse;
    // Query rows.  Prefill: one work item per query head, rows are tokens.
    // Step: the G query heads of a KV group are packed into one row space,
    // row p = t * G + hh for token t and head kvh * G + hh, so small blocks
    // still fill the query tiles; nrows = G * Lq rows per (b, KV head).
    // split-KV partials (step only), in blocks of 32 packed rows (nrb =
    // ceil(G * Lq / 32) blocks per (b, KV head)).  f32 output: o
    // [S][B][Hkv][nrb][D/4][64 lanes][4] f32 unnormalised, in the
    // accumulator's register order, and (m, l) [S][B][Hkv][nrb * 32][2].
    // bf16 output: o / l as bf16 [S][B][Hkv][nrb][D/8][64 lanes][8] in
    // register order (two accumulator groups per lane) and m + log2(l)
    // [S][B][Hkv][nrb * 32] f32 at part_ml.
    float *part_o, *part_ml;
    int32_t nrb;
    int32_t nrows;       // rows per item's head space: Lq (prefill) or G * Lq (step)
    int32_t gi;          // work items per (b, KV head, q-tile, split): G (prefill) or 1 (step)
    int32_t B, Lq, Hq, Hkv, G;
    int32_t mode;        // MODE_PREFILL or MODE_STEP
    int32_t paged;       // prefill only: keys/values come from the pool
    int32_t fuse_append; // step only: also commit kc/vc to the pool
    int32_t nsplit;      // KV splits per query tile (1 in the prefill)
    int32_t nqt;         // query tiles per head space: of Lq rows (prefill) or G * Lq packed rows (step)
    int32_t n_work;      // B * Hkv * gi * nqt * nsplit
    int32_t per_xcd;     // ceil(n_work / 8)
    int32_t per_group;   // gi * nqt * nsplit: work items per (b, KV head)
    int32_t per_qt;      // gi * nsplit: work items per (b, KV head, q-tile)
    // dividers by per_group, per_qt, G, Hkv and nsplit
    FastDiv fd_group, fd_qt, fd_g, fd_hkv, fd_split;
    FastDiv fd_gq;       // divider by G (packed row -> token)
    FastDiv fd_b;        // divider by B (step groups taken KV-head-major)
    float scale_log2;    // scale * log2(e)
    // step: cache lengths (and segment starts) also passed by value when
    // batch <= LENS_IN_ARGS, so the first page lookup does not wait on a load
    // of them
    int32_t lens_in_args;
    int32_t lens_arg[32];
    int32_t text_arg[32];   // step: segment starts by value (new_len: none)
    int32_t nl_arg[32];     // step: new-block lengths by value
};

constexpr int LENS_IN_ARGS = 32;

struct AppendArgs {
    const uint16_t *kn, *vn;
    int64_t kn_sb, kn_st, kn_sh;
    int64_t vn_sb, vn_st, vn_sh;
    uint16_t *kpool, *vpool;
    const int32_t *page_table;
    int32_t max_pages;
    const int32_t *cache_lens;
    const int32_t *new_lens;   // NULL: every stream commits Ln tokens
    int32_t B, Ln, Hkv, D;
};

// Gradients of the whole-sequence path (contiguous K/V).  bf16 inputs,
// f32 gradients; element strides.
struct BwdArgs {
    const uint16_t *q, *k, *v, *o, *dout;
    int64_t q_sb, q_st, q_sh;
    int64_t k_sb, k_st, k_sh;
    int64_t v_sb, v_st, v_sh;
    int64_t o_sb, o_st, o_sh;
    int64_t do_sb, do_st, do_sh;
    const float *lse;            // forward lse [B][Hq][L] (natural log)
    const int32_t *offsets;      // [B][nb+1]
    const int32_t *text_starts;  // [B][nb] or nullptr
    int32_t nb;
    float *dq, *dk, *dv;
    int64_t dq_sb, dq_st, dq_sh;
    int64_t dk_sb, dk_st, dk_sh;
    int64_t dv_sb, dv_st, dv_sh;
    // workspace: per row (lse * log2(e), rowsum(dO * O)) [B][Hq][L], and the
    // end of the keys each token sees [B][L]
    float *dl;
    int32_t *kend;
    int32_t B, L, Hq, Hkv, G;
    float scale, scale_log2;
};

// Launch shapes compiled into the library.
struct TileShape {
    int nb;  // 32-query column blocks per wave
    int nw;  // waves per work-group
    int qtile() const { return nb * nw * 32; }
    // work-groups resident per CU (LDS and registers allow one)
    int groups_per_cu() const { return 1; }
};

// Each returns 0 or a HIP error code (hipError_t as int).
int launch_attention(const AttnArgs &a, int head_dim, TileShape shape, void *stream);
int launch_combine(const AttnArgs &a, int head_dim, void *stream);
int launch_append(const AppendArgs &a, void *stream);
// prep (row sums, key ends), then dQ and dK/dV; 0 or a HIP error code
int launch_prefill_bwd(const BwdArgs &a, int head_dim, void *stream);
// Compute units of the current HIP device (queried once per device, then
// cached): 0 and *cus set, or a HIP error code (e.g. no device).
int current_device_cus(int *cus);

// Bytes of the per-device scratch array behind the allocation-free step.
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)32 << 20;
// Device address of the current device's scratch array (looked up once per
// device): 0 and *ptr set, or a HIP error code.
int scratch_address(void **ptr);

}  // namespace ws
