// C ABI of libwsattn: host-side validation and launch planning.
//
// Plain C++ (no HIP headers): every argument is checked here before any
// device work is enqueued, so a rejected call leaves all device memory
// untouched.  Kernels are reached through the launchers of ws_kernels.hip.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "../../include/ws_attn.h"
#include "ws_kernels.h"

namespace {

thread_local char g_err[512];

int fail(int status, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return status;
}

int ok() {
    g_err[0] = '\0';
    return WS_OK;
}

constexpr int WS_MAX_SPLITS = ws::MAX_SPLITS;
static_assert(WS_NOALLOC_SCRATCH_BYTES == ws::NOALLOC_SCRATCH_BYTES, "one scratch size");
// packed query rows of one (stream, KV head) in a step: G x new_len (the
// kernels index them in 32-bit arithmetic)
constexpr int64_t WS_MAX_STEP_ROWS = ((int64_t)1 << 30);
constexpr int WS_MAX_HEAD_DIM = 128;

int env_int(const char *name, int dflt) {
    const char *s = std::getenv(name);
    if (!s || !*s) return dflt;
    return std::atoi(s);
}

// Tuning override of the KV split count (WS_SPLITS = 1..32), read once, at
// the first call that plans a step, and fixed for the rest of the process,
// so workspace queries and calls always agree.  0: no override.
int split_override() {
    static const int s = [] {
        const int v = env_int("WS_SPLITS", 0);
        return v <= 0 ? 0 : v > WS_MAX_SPLITS ? WS_MAX_SPLITS : v;
    }();
    return s;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// Token stride limit of key/value tensors (elements): the kernels form the
// offsets of one 64-key tile's rows in 32 bits.
constexpr int64_t WS_MAX_KV_TOKEN_STRIDE = (int64_t)1 << 24;

// Checks pointer, dtype, alignment and strides of one token tensor.
int check_tensor(const char *name, const ws_tensor4 &t, bool allow_f32) {
    if (!t.ptr) return fail(WS_ERR_NULL, "%s.ptr is NULL", name);
    if (t.dtype != WS_DTYPE_BF16 && !(allow_f32 && t.dtype == WS_DTYPE_F32))
        return fail(WS_ERR_UNSUPPORTED, "%s.dtype %d not supported", name, (int)t.dtype);
    if (t.stride_b < 0 || t.stride_t < 0 || t.stride_h < 0)
        return fail(WS_ERR_SHAPE, "%s has a negative stride", name);
    const int64_t q = (t.dtype == WS_DTYPE_BF16) ? 8 : 4;  // elements per 16 bytes
    if (!aligned16(t.ptr) || t.stride_b % q || t.stride_t % q || t.stride_h % q)
        return fail(WS_ERR_ALIGN, "%s: pointer must be 16-byte aligned and strides multiples of 16 bytes", name);
    return WS_OK;
}

int check_kv_tensor(const char *name, const ws_tensor4 &t) {
    if (int rc = check_tensor(name, t, false)) return rc;
    if (t.stride_t >= WS_MAX_KV_TOKEN_STRIDE)
        return fail(WS_ERR_SHAPE, "%s token stride %lld must be below %lld elements", name,
                    (long long)t.stride_t, (long long)WS_MAX_KV_TOKEN_STRIDE);
    return WS_OK;
}

int check_head_dim(int d) {
    if (d != 64 && d != 128) return fail(WS_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", d);
    return WS_OK;
}

int check_paged(const ws_paged_kv *kv) {
    if (!kv) return fail(WS_ERR_NULL, "kv is NULL");
    if (!kv->k_pool || !kv->v_pool) return fail(WS_ERR_NULL, "kv pool pointer is NULL");
    if (!kv->page_table_dev || !kv->page_table_host) return fail(WS_ERR_NULL, "kv page table pointer is NULL");
    if (kv->num_pages <= 0 || kv->max_pages_per_seq < 0 || kv->num_kv_heads <= 0)
        return fail(WS_ERR_SHAPE, "kv: num_pages %d, max_pages_per_seq %d, num_kv_heads %d",
                    (int)kv->num_pages, (int)kv->max_pages_per_seq, (int)kv->num_kv_heads);
    if (kv->page_size != WS_PAGE_SIZE)
        return fail(WS_ERR_UNSUPPORTED, "page_size %d not supported (only %d)", (int)kv->page_size, WS_PAGE_SIZE);
    if (int rc = check_head_dim(kv->head_dim)) return rc;
    if (!aligned16(kv->k_pool) || !aligned16(kv->v_pool))
        return fail(WS_ERR_ALIGN, "kv pools must be 16-byte aligned");
    return WS_OK;
}

// Every page that positions [0, n) of stream b live in must exist.
int check_pages(const ws_paged_kv *kv, int b, int64_t n) {
    if (n > (int64_t)kv->max_pages_per_seq * kv->page_size)
        return fail(WS_ERR_CAPACITY, "stream %d needs %lld tokens but holds at most %lld", b,
                    (long long)n, (long long)kv->max_pages_per_seq * kv->page_size);
    const int64_t pages = (n + kv->page_size - 1) / kv->page_size;
    const int32_t *row = kv->page_table_host + (int64_t)b * kv->max_pages_per_seq;
    for (int64_t p = 0; p < pages; ++p)
        if (row[p] < 0 || row[p] >= kv->num_pages)
            return fail(WS_ERR_PAGE, "page_table[%d][%lld] = %d outside [0, %d)", b, (long long)p,
                        (int)row[p], (int)kv->num_pages);
    return WS_OK;
}

struct StepPlan {
    ws::TileShape shape;
    int nqt;
    int nsplit;
};

// Query tile and KV split count of a streaming step.
// One launch shape: 8 waves x 32 query rows (256-query tiles).
ws::TileShape default_shape() { return ws::TileShape{1, 8}; }

// Per-item fixed cost (prologue, epilogue, partial stores) in units of one
// 64-key tile of the loop, for the split model below.
constexpr int64_t SPLIT_FIXED_TILES = 4;

// The step packs the G query heads of a KV group into one row space of
// G * lq rows (see AttnArgs).  Split count: by default the largest that
// still fits the work-groups in one round on the CUs (every split keeps at
// least two 64-key tiles).  A round-count model, rounds(s) x (tiles per
// split + fixed cost), minimised with a bias to fewer splits, replaces it
// when it predicts a gain of more than 10 %:
// when the items do not fill the last round (a batch of 3 or 5 long
// streams, or new blocks of different lengths, nl != NULL, whose tiles of
// padding only do no work).
StepPlan plan_step(int num_cus, int batch, int hq, int hkv, int lq, int64_t max_k, const int32_t *nl = nullptr) {
    StepPlan p;
    p.shape = default_shape();
    const int64_t qt = p.shape.qtile();
    const int64_t G = hq / hkv;
    p.nqt = (int)((G * lq + qt - 1) / qt);
    // work items with at least one real row, per split
    int64_t base = (int64_t)batch * hkv * p.nqt;
    if (nl) {
        base = 0;
        for (int b = 0; b < batch; ++b) base += (G * nl[b] + qt - 1) / qt;
        base *= hkv;
    }
    const int64_t ntiles = (max_k + 63) / 64;
    const int64_t slots = (int64_t)num_cus * p.shape.groups_per_cu();
    int64_t cap = ntiles / 2;
    if (cap > WS_MAX_SPLITS) cap = WS_MAX_SPLITS;
    if (cap < 1) cap = 1;
    int64_t ns = (base > 0 && base < slots) ? slots / base : 1;
    if (ns > cap) ns = cap;
    // real q-tiles of the streams before stream b (nl only)
    std::vector<int64_t> pre(nl ? batch + 1 : 0);
    if (nl)
        for (int b = 0; b < batch; ++b) pre[b + 1] = pre[b] + (G * nl[b] + qt - 1) / qt;
    // rounds of work-groups x (tiles per split + fixed cost)
    auto cost = [&](int64_t s) -> int64_t {
        const int64_t per_split = (ntiles + s - 1) / s + SPLIT_FIXED_TILES;
        if (!nl) return (base * s + slots - 1) / slots * per_split;
        // Items of padding only finish at once, so rounds are counted per
        // XCD, from the real items in its range of the launch order: groups
        // KV-head-major (g = kvh * batch + b), P = nqt * s items per group,
        // of which the first (real tiles of b) * s are real.
        const int64_t P = (int64_t)p.nqt * s, n_work = (int64_t)batch * hkv * P;
        const int64_t per = (n_work + ws::NUM_XCD - 1) / ws::NUM_XCD;
        auto real_before = [&](int64_t w) -> int64_t {   // real items in [0, w)
            if (w >= n_work) return hkv * pre[batch] * s;
            const int64_t g = w / P, kvh = g / batch, b = g % batch;
            return (kvh * pre[batch] + pre[b]) * s + std::min(w - g * P, (pre[b + 1] - pre[b]) * s);
        };
        const int64_t per_cu = std::max<int64_t>(1, slots / ws::NUM_XCD);
        int64_t rounds = 0;
        for (int64_t x = 0; x < ws::NUM_XCD; ++x) {
            const int64_t c = real_before((x + 1) * per) - real_before(x * per);
            rounds = std::max(rounds, (c + per_cu - 1) / per_cu);
        }
        return rounds * per_split;
    };
    if (base > 0) {
        // the fewest splits within 2 % of the modelled minimum (each split
        // adds merge work and thins the L2 reuse of a KV range across q-tiles,
        // which the model leaves out)
        int64_t lo = cost(1);
        for (int64_t s = 2; s <= cap; ++s) lo = std::min(lo, cost(s));
        int64_t best = 1;
        while (50 * cost(best) > 51 * lo) ++best;
        if (10 * cost(best) < 9 * cost(ns)) ns = best;
    }
    if (const int s_ov = split_override()) ns = s_ov;
    p.nsplit = (int)ns;
    return p;
}

// Partials are kept in blocks of 32 packed rows per (stream, KV head).
size_t step_workspace(const StepPlan &p, int batch, int hq, int hkv, int lq) {
    if (p.nsplit <= 1) return 0;
    const size_t rows = ((size_t)(hq / hkv) * lq + 31) / 32 * 32;
    return (size_t)p.nsplit * batch * hkv * rows * (WS_MAX_HEAD_DIM + 2) * sizeof(float);
}

ws::TileShape plan_prefill(int) { return default_shape(); }

// Backward workspace: (lse * log2 e, <dO, O>) per row as f32 pairs, then the
// key end of each token (int32), at a 256-byte aligned offset.
size_t bwd_dl_bytes(int batch, int hq, int seq) {
    return ((size_t)batch * hq * seq * 2 * sizeof(float) + 255) / 256 * 256;
}
size_t bwd_workspace(int batch, int hq, int seq) {
    return bwd_dl_bytes(batch, hq, seq) + (size_t)batch * seq * sizeof(int32_t);
}

// Total work items; fails when the grid would not fit the kernel's int math.
bool finish_work(ws::AttnArgs &a) {
    const int64_t n = (int64_t)a.B * a.Hkv * a.gi * a.nqt * a.nsplit;
    if (n > (int64_t)1 << 30) return false;
    a.n_work = (int32_t)n;
    a.per_xcd = (a.n_work + ws::NUM_XCD - 1) / ws::NUM_XCD;
    a.per_qt = a.gi * a.nsplit;
    a.per_group = a.per_qt * a.nqt;
    a.fd_group = ws::fastdiv_make((uint32_t)a.per_group);
    a.fd_qt = ws::fastdiv_make((uint32_t)a.per_qt);
    a.fd_g = ws::fastdiv_make((uint32_t)a.gi);
    a.fd_gq = ws::fastdiv_make((uint32_t)a.G);
    a.fd_hkv = ws::fastdiv_make((uint32_t)a.Hkv);
    a.fd_split = ws::fastdiv_make((uint32_t)a.nsplit);
    a.fd_b = ws::fastdiv_make((uint32_t)a.B);
    return true;
}

int step_impl(ws_tensor4 q, ws_tensor4 k_new, ws_tensor4 v_new, const ws_paged_kv *kv,
              const int32_t *cache_lens_host, const int32_t *cache_lens_dev,
              const int32_t *nl_host, const int32_t *nl_dev,
              const int32_t *text_host, const int32_t *text_dev, int32_t batch,
              int32_t new_len, int32_t num_q_heads, float scale, int32_t flags,
              ws_tensor4 out, float *lse, void *workspace, size_t workspace_bytes,
              void *stream, bool noalloc = false);
int append_impl(const ws_paged_kv *kv, int32_t batch, const int32_t *cache_lens_host,
                const int32_t *cache_lens_dev, const int32_t *nl_host, const int32_t *nl_dev, int32_t new_len,
                ws_tensor4 k_new, ws_tensor4 v_new, void *stream);
int prefill_impl(ws_tensor4 q, ws_tensor4 k, ws_tensor4 v, const ws_paged_kv *kv_or_null,
                 const int32_t *block_offsets_host, const int32_t *block_offsets_dev,
                 const int32_t *text_host, const int32_t *text_dev,
                 int32_t batch, int32_t seq_len, int32_t num_blocks, int32_t num_q_heads,
                 int32_t num_kv_heads, int32_t head_dim, float scale, ws_tensor4 out,
                 float *lse, void *stream);

}  // namespace

extern "C" {

int ws_abi_version(void) { return WS_ABI_VERSION; }

const char *ws_status_string(int status) {
    switch (status) {
        case WS_OK: return "WS_OK";
        case WS_ERR_NULL: return "WS_ERR_NULL";
        case WS_ERR_SHAPE: return "WS_ERR_SHAPE";
        case WS_ERR_UNSUPPORTED: return "WS_ERR_UNSUPPORTED";
        case WS_ERR_ALIGN: return "WS_ERR_ALIGN";
        case WS_ERR_OFFSETS: return "WS_ERR_OFFSETS";
        case WS_ERR_PAGE: return "WS_ERR_PAGE";
        case WS_ERR_CAPACITY: return "WS_ERR_CAPACITY";
        case WS_ERR_HEADS: return "WS_ERR_HEADS";
        case WS_ERR_WORKSPACE: return "WS_ERR_WORKSPACE";
        case WS_ERR_HIP: return "WS_ERR_HIP";
        default: return "WS_ERR_UNKNOWN";
    }
}

const char *ws_last_error(void) { return g_err; }

size_t ws_workspace_bytes(int32_t op, int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                          int32_t max_q, int32_t max_k) {
    if (op == WS_OP_PREFILL_BWD) {
        if (batch <= 0 || num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads || max_q <= 0)
            return 0;
        return bwd_workspace(batch, num_q_heads, max_q);
    }
    if (op != WS_OP_STEP) return 0;
    if (batch <= 0 || num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads || max_q <= 0 ||
        max_k < max_q)
        return 0;
    if ((int64_t)(num_q_heads / num_kv_heads) * max_q > WS_MAX_STEP_ROWS) return 0;
    int cus = 0;
    if (ws::current_device_cus(&cus)) return 0;
    const StepPlan p = plan_step(cus, batch, num_q_heads, num_kv_heads, max_q, max_k);
    return step_workspace(p, batch, num_q_heads, num_kv_heads, max_q);
}

size_t ws_step_workspace_bytes_varlen(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t new_len,
                                      const int32_t *cache_lens_host, const int32_t *new_lens_host) {
    if (batch <= 0 || num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads || new_len <= 0 ||
        !cache_lens_host || !new_lens_host)
        return 0;
    if ((int64_t)(num_q_heads / num_kv_heads) * new_len > WS_MAX_STEP_ROWS) return 0;
    int64_t max_k = 0;
    for (int b = 0; b < batch; ++b) {
        if (cache_lens_host[b] < 0 || new_lens_host[b] < 1 || new_lens_host[b] > new_len) return 0;
        const int64_t k = (int64_t)cache_lens_host[b] + new_lens_host[b];
        if (k > max_k) max_k = k;
    }
    if (max_k > INT32_MAX) return 0;
    int cus = 0;
    if (ws::current_device_cus(&cus)) return 0;
    const StepPlan p = plan_step(cus, batch, num_q_heads, num_kv_heads, new_len, max_k, new_lens_host);
    return step_workspace(p, batch, num_q_heads, num_kv_heads, new_len);
}

int ws_step_plan(int32_t num_cus, int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t new_len,
                 const int32_t *cache_lens_host, const int32_t *new_lens_host, int32_t *num_splits,
                 size_t *workspace_bytes) {
    if (!cache_lens_host || !num_splits || !workspace_bytes) return fail(WS_ERR_NULL, "NULL argument");
    if (num_cus < 0 || batch <= 0 || new_len <= 0 || num_q_heads <= 0 || num_kv_heads <= 0)
        return fail(WS_ERR_SHAPE, "num_cus %d, batch %d, new_len %d, heads %d/%d", (int)num_cus, (int)batch,
                    (int)new_len, (int)num_q_heads, (int)num_kv_heads);
    if (num_q_heads % num_kv_heads)
        return fail(WS_ERR_HEADS, "num_q_heads %d not a multiple of num_kv_heads %d", (int)num_q_heads,
                    (int)num_kv_heads);
    if ((int64_t)(num_q_heads / num_kv_heads) * new_len > WS_MAX_STEP_ROWS)
        return fail(WS_ERR_SHAPE, "new_len x query heads per KV head exceeds %lld", (long long)WS_MAX_STEP_ROWS);
    int64_t max_k = 0;
    for (int b = 0; b < batch; ++b) {
        if (cache_lens_host[b] < 0) return fail(WS_ERR_SHAPE, "cache_lens[%d] = %d", b, (int)cache_lens_host[b]);
        if (new_lens_host && (new_lens_host[b] < 1 || new_lens_host[b] > new_len))
            return fail(WS_ERR_SHAPE, "new_lens[%d] = %d outside [1, new_len %d]", b, (int)new_lens_host[b],
                        (int)new_len);
        max_k = std::max(max_k, (int64_t)cache_lens_host[b] + (new_lens_host ? new_lens_host[b] : new_len));
    }
    if (max_k > INT32_MAX) return fail(WS_ERR_SHAPE, "too many keys");
    int cus = num_cus;
    if (cus == 0)
        if (int e = ws::current_device_cus(&cus)) return fail(WS_ERR_HIP, "no device to plan for (hip error %d)", e);
    const StepPlan p = plan_step(cus, batch, num_q_heads, num_kv_heads, new_len, max_k, new_lens_host);
    *num_splits = p.nsplit;
    *workspace_bytes = step_workspace(p, batch, num_q_heads, num_kv_heads, new_len);
    return ok();
}

int ws_kv_append(const ws_paged_kv *kv, int32_t batch, const int32_t *cache_lens_host,
                 const int32_t *cache_lens_dev, int32_t new_len, ws_tensor4 k_new, ws_tensor4 v_new,
                 void *stream) {
    return append_impl(kv, batch, cache_lens_host, cache_lens_dev, nullptr, nullptr, new_len, k_new, v_new, stream);
}

int ws_kv_append_varlen(const ws_paged_kv *kv, int32_t batch, const int32_t *cache_lens_host,
                        const int32_t *cache_lens_dev, const int32_t *new_lens_host, const int32_t *new_lens_dev,
                        int32_t new_len, ws_tensor4 k_new, ws_tensor4 v_new, void *stream) {
    if (!new_lens_host || !new_lens_dev) return fail(WS_ERR_NULL, "new_lens pointer is NULL");
    return append_impl(kv, batch, cache_lens_host, cache_lens_dev, new_lens_host, new_lens_dev, new_len, k_new,
                       v_new, stream);
}

int ws_block_causal_attn_fwd(ws_tensor4 q, ws_tensor4 k_new, ws_tensor4 v_new, const ws_paged_kv *kv,
                             const int32_t *cache_lens_host, const int32_t *cache_lens_dev, int32_t batch,
                             int32_t new_len, int32_t num_q_heads, float scale, int32_t flags,
                             ws_tensor4 out, float *lse, void *workspace, size_t workspace_bytes,
                             void *stream) {
    return step_impl(q, k_new, v_new, kv, cache_lens_host, cache_lens_dev, nullptr, nullptr, nullptr, nullptr, batch,
                     new_len, num_q_heads, scale, flags, out, lse, workspace, workspace_bytes, stream);
}

int ws_block_causal_attn_fwd_noalloc(ws_tensor4 q, ws_tensor4 k_new, ws_tensor4 v_new, const ws_paged_kv *kv,
                                     const int32_t *cache_lens_host, const int32_t *cache_lens_dev, int32_t batch,
                                     int32_t new_len, int32_t num_q_heads, float scale, int32_t flags,
                                     ws_tensor4 out, float *lse, void *stream) {
    return step_impl(q, k_new, v_new, kv, cache_lens_host, cache_lens_dev, nullptr, nullptr, nullptr, nullptr, batch,
                     new_len, num_q_heads, scale, flags, out, lse, nullptr, 0, stream, true);
}

int ws_block_causal_attn_fwd_text(ws_tensor4 q, ws_tensor4 k_new, ws_tensor4 v_new, const ws_paged_kv *kv,
                                  const int32_t *cache_lens_host, const int32_t *cache_lens_dev,
                                  const int32_t *text_starts_host, const int32_t *text_starts_dev,
                                  int32_t batch, int32_t new_len, int32_t num_q_heads, float scale, int32_t flags,
                                  ws_tensor4 out, float *lse, void *workspace, size_t workspace_bytes,
                                  void *stream) {
    if (!text_starts_host || !text_starts_dev) return fail(WS_ERR_NULL, "text_starts pointer is NULL");
    return step_impl(q, k_new, v_new, kv, cache_lens_host, cache_lens_dev, nullptr, nullptr, text_starts_host,
                     text_starts_dev, batch, new_len, num_q_heads, scale, flags, out, lse, workspace,
                     workspace_bytes, stream);
}

int ws_block_causal_attn_fwd_varlen(ws_tensor4 q, ws_tensor4 k_new, ws_tensor4 v_new, const ws_paged_kv *kv,
                                    const int32_t *cache_lens_host, const int32_t *cache_lens_dev,
                                    const int32_t *new_lens_host, const int32_t *new_lens_dev,
                                    const int32_t *text_starts_host, const int32_t *text_starts_dev,
                                    int32_t batch, int32_t new_len, int32_t num_q_heads, float scale,
                                    int32_t flags, ws_tensor4 out, float *lse, void *workspace,
                                    size_t workspace_bytes, void *stream) {
    if (!new_lens_host || !new_lens_dev) return fail(WS_ERR_NULL, "new_lens pointer is NULL");
    if (!text_starts_host != !text_starts_dev) return fail(WS_ERR_NULL, "text_starts: give both copies or neither");
    return step_impl(q, k_new, v_new, kv, cache_lens_host, cache_lens_dev, new_lens_host, new_lens_dev,
                     text_starts_host, text_starts_dev, batch, new_len, num_q_heads, scale, flags, out, lse,
                     workspace, workspace_bytes, stream);
}

int ws_block_causal_prefill(ws_tensor4 q, ws_tensor4 k, ws_tensor4 v, const ws_paged_kv *kv_or_null,
                            const int32_t *block_offsets_host, const int32_t *block_offsets_dev,
                            int32_t batch, int32_t seq_len, int32_t num_blocks, int32_t num_q_heads,
                            int32_t num_kv_heads, int32_t head_dim, float scale, ws_tensor4 out,
                            float *lse, void *stream) {
    return prefill_impl(q, k, v, kv_or_null, block_offsets_host, block_offsets_dev, nullptr, nullptr, batch,
                        seq_len, num_blocks, num_q_heads, num_kv_heads, head_dim, scale, out, lse, stream);
}

int ws_block_causal_prefill_text(ws_tensor4 q, ws_tensor4 k, ws_tensor4 v, const ws_paged_kv *kv_or_null,
                                 const int32_t *block_offsets_host, const int32_t *block_offsets_dev,
                                 const int32_t *text_starts_host, const int32_t *text_starts_dev,
                                 int32_t batch, int32_t seq_len, int32_t num_blocks, int32_t num_q_heads,
                                 int32_t num_kv_heads, int32_t head_dim, float scale, ws_tensor4 out,
                                 float *lse, void *stream) {
    if (!text_starts_host || !text_starts_dev) return fail(WS_ERR_NULL, "text_starts pointer is NULL");
    return prefill_impl(q, k, v, kv_or_null, block_offsets_host, block_offsets_dev, text_starts_host,
                        text_starts_dev, batch, seq_len, num_blocks, num_q_heads, num_kv_heads, head_dim,
                        scale, out, lse, stream);
}

int ws_block_causal_prefill_bwd(ws_tensor4 q, ws_tensor4 k, ws_tensor4 v, ws_tensor4 o, ws_tensor4 dout,
                                const float *lse, const int32_t *block_offsets_host,
                                const int32_t *block_offsets_dev, const int32_t *text_starts_host,
                                const int32_t *text_starts_dev, int32_t batch, int32_t seq_len, int32_t num_blocks,
                                int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, float scale,
                                ws_tensor4 dq, ws_tensor4 dk, ws_tensor4 dv, void *workspace,
                                size_t workspace_bytes, void *stream) {
    if (batch < 0 || seq_len < 0 || num_blocks < 0 || num_q_heads <= 0 || num_kv_heads <= 0)
        return fail(WS_ERR_SHAPE, "batch %d, seq_len %d, num_blocks %d, heads %d/%d", (int)batch, (int)seq_len,
                    (int)num_blocks, (int)num_q_heads, (int)num_kv_heads);
    if (batch == 0 || seq_len == 0) return ok();
    if (int rc = check_tensor("q", q, false)) return rc;
    if (int rc = check_tensor("k", k, false)) return rc;
    if (int rc = check_tensor("v", v, false)) return rc;
    if (int rc = check_tensor("o", o, false)) return rc;
    if (int rc = check_tensor("dout", dout, false)) return rc;
    if (int rc = check_tensor("dq", dq, true)) return rc;
    if (int rc = check_tensor("dk", dk, true)) return rc;
    if (int rc = check_tensor("dv", dv, true)) return rc;
    if (dq.dtype != WS_DTYPE_F32 || dk.dtype != WS_DTYPE_F32 || dv.dtype != WS_DTYPE_F32)
        return fail(WS_ERR_UNSUPPORTED, "dq, dk and dv must be f32");
    if (!lse) return fail(WS_ERR_NULL, "lse is NULL");
    if ((uintptr_t)lse & 3u) return fail(WS_ERR_ALIGN, "lse must be 4-byte aligned");
    if (!block_offsets_host || !block_offsets_dev) return fail(WS_ERR_NULL, "block offsets pointer is NULL");
    if (!text_starts_host != !text_starts_dev) return fail(WS_ERR_NULL, "text_starts: give both copies or neither");
    if (int rc = check_head_dim(head_dim)) return rc;
    if (!(scale > 0.f) || !std::isfinite(scale)) return fail(WS_ERR_UNSUPPORTED, "scale must be finite and > 0");
    if (num_q_heads % num_kv_heads)
        return fail(WS_ERR_HEADS, "num_q_heads %d not a multiple of num_kv_heads %d", (int)num_q_heads,
                    (int)num_kv_heads);
    for (int b = 0; b < batch; ++b) {
        const int32_t *off = block_offsets_host + (int64_t)b * (num_blocks + 1);
        if (off[0] != 0) return fail(WS_ERR_OFFSETS, "block_offsets[%d][0] = %d, must be 0", b, (int)off[0]);
        for (int n = 0; n < num_blocks; ++n) {
            if (off[n + 1] < off[n])
                return fail(WS_ERR_OFFSETS, "block_offsets[%d] decreases at %d", b, n + 1);
            if (text_starts_host) {
                const int32_t t = text_starts_host[(int64_t)b * num_blocks + n];
                if (t < off[n] || t > off[n + 1])
                    return fail(WS_ERR_OFFSETS, "text_starts[%d][%d] = %d outside block [%d, %d]", b, n, (int)t,
                                (int)off[n], (int)off[n + 1]);
            }
        }
        if (off[num_blocks] != seq_len)
            return fail(WS_ERR_OFFSETS, "block_offsets[%d][%d] = %d, must equal seq_len %d", b, (int)num_blocks,
                        (int)off[num_blocks], (int)seq_len);
    }
    const int64_t work = (int64_t)batch * num_q_heads * ((seq_len + 127) / 128);
    if (work > INT32_MAX) return fail(WS_ERR_SHAPE, "too many work items");
    const size_t need = bwd_workspace(batch, num_q_heads, seq_len);
    if (!workspace || workspace_bytes < need || !aligned16(workspace))
        return fail(WS_ERR_WORKSPACE, "workspace needs %zu bytes (16-byte aligned), got %zu", need,
                    workspace ? workspace_bytes : (size_t)0);
    ws::BwdArgs a{};
    a.q = (const uint16_t *)q.ptr; a.q_sb = q.stride_b; a.q_st = q.stride_t; a.q_sh = q.stride_h;
    a.k = (const uint16_t *)k.ptr; a.k_sb = k.stride_b; a.k_st = k.stride_t; a.k_sh = k.stride_h;
    a.v = (const uint16_t *)v.ptr; a.v_sb = v.stride_b; a.v_st = v.stride_t; a.v_sh = v.stride_h;
    a.o = (const uint16_t *)o.ptr; a.o_sb = o.stride_b; a.o_st = o.stride_t; a.o_sh = o.stride_h;
    a.dout = (const uint16_t *)dout.ptr; a.do_sb = dout.stride_b; a.do_st = dout.stride_t; a.do_sh = dout.stride_h;
    a.lse = lse;
    a.offsets = block_offsets_dev;
    a.text_starts = text_starts_dev;
    a.nb = num_blocks;
    a.dq = (float *)dq.ptr; a.dq_sb = dq.stride_b; a.dq_st = dq.stride_t; a.dq_sh = dq.stride_h;
    a.dk = (float *)dk.ptr; a.dk_sb = dk.stride_b; a.dk_st = dk.stride_t; a.dk_sh = dk.stride_h;
    a.dv = (float *)dv.ptr; a.dv_sb = dv.stride_b; a.dv_st = dv.stride_t; a.dv_sh = dv.stride_h;
    a.dl = (float *)workspace;
    a.kend = (int32_t *)((char *)workspace + bwd_dl_bytes(batch, num_q_heads, seq_len));
    a.B = batch; a.L = seq_len; a.Hq = num_q_heads; a.Hkv = num_kv_heads; a.G = num_q_heads / num_kv_heads;
    a.scale = scale;
    a.scale_log2 = scale * 1.4426950408889634f;
    if (int e = ws::launch_prefill_bwd(a, head_dim, stream))
        return fail(WS_ERR_HIP, "backward launch failed (hip error %d)", e);
    return ok();
}

}  // extern "C"

namespace {

// Commit new tokens to the cache (nl_* NULL: new_len tokens per stream).
int append_impl(const ws_paged_kv *kv, int32_t batch, const int32_t *cache_lens_host,
                const int32_t *cache_lens_dev, const int32_t *nl_host, const int32_t *nl_dev, int32_t new_len,
                ws_tensor4 k_new, ws_tensor4 v_new, void *stream) {
    if (int rc = check_paged(kv)) return rc;
    if (!cache_lens_host || !cache_lens_dev) return fail(WS_ERR_NULL, "cache_lens pointer is NULL");
    if (batch < 0 || new_len < 0) return fail(WS_ERR_SHAPE, "batch %d, new_len %d", (int)batch, (int)new_len);
    if (batch == 0 || new_len == 0) return ok();  // nothing is read or written
    if (int rc = check_tensor("k_new", k_new, false)) return rc;
    if (int rc = check_tensor("v_new", v_new, false)) return rc;
    for (int b = 0; b < batch; ++b) {
        if (cache_lens_host[b] < 0) return fail(WS_ERR_SHAPE, "cache_lens[%d] = %d", b, (int)cache_lens_host[b]);
        if (nl_host && (nl_host[b] < 0 || nl_host[b] > new_len))
            return fail(WS_ERR_SHAPE, "new_lens[%d] = %d outside [0, new_len %d]", b, (int)nl_host[b], (int)new_len);
        if (int rc = check_pages(kv, b, (int64_t)cache_lens_host[b] + (nl_host ? nl_host[b] : new_len))) return rc;
    }
    ws::AppendArgs a{};
    a.kn = (const uint16_t *)k_new.ptr;
    a.vn = (const uint16_t *)v_new.ptr;
    a.kn_sb = k_new.stride_b; a.kn_st = k_new.stride_t; a.kn_sh = k_new.stride_h;
    a.vn_sb = v_new.stride_b; a.vn_st = v_new.stride_t; a.vn_sh = v_new.stride_h;
    a.kpool = (uint16_t *)kv->k_pool;
    a.vpool = (uint16_t *)kv->v_pool;
    a.page_table = kv->page_table_dev;
    a.max_pages = kv->max_pages_per_seq;
    a.cache_lens = cache_lens_dev;
    a.new_lens = nl_host ? nl_dev : nullptr;
    a.B = batch; a.Ln = new_len; a.Hkv = kv->num_kv_heads; a.D = kv->head_dim;
    if (int e = ws::launch_append(a, stream)) return fail(WS_ERR_HIP, "append launch failed (hip error %d)", e);
    return ok();
}

// One streaming step (text_* NULL: no token-causal segment; nl_* NULL:
// every new block holds new_len tokens).
int step_impl(ws_tensor4 q, ws_tensor4 k_new, ws_tensor4 v_new, const ws_paged_kv *kv,
              const int32_t *cache_lens_host, const int32_t *cache_lens_dev,
              const int32_t *nl_host, const int32_t *nl_dev,
              const int32_t *text_host, const int32_t *text_dev, int32_t batch,
              int32_t new_len, int32_t num_q_heads, float scale, int32_t flags,
              ws_tensor4 out, float *lse, void *workspace, size_t workspace_bytes,
              void *stream, bool noalloc) {
    if (int rc = check_paged(kv)) return rc;
    if (!cache_lens_host || !cache_lens_dev) return fail(WS_ERR_NULL, "cache_lens pointer is NULL");
    if (batch < 0 || new_len < 0 || num_q_heads <= 0)
        return fail(WS_ERR_SHAPE, "batch %d, new_len %d, num_q_heads %d", (int)batch, (int)new_len, (int)num_q_heads);
    if (batch == 0 || new_len == 0) return ok();  // no query row: nothing is read or written
    if (int rc = check_tensor("q", q, false)) return rc;
    if (int rc = check_kv_tensor("k_new", k_new)) return rc;
    if (int rc = check_kv_tensor("v_new", v_new)) return rc;
    if (int rc = check_tensor("out", out, true)) return rc;
    if (flags & ~WS_FUSE_APPEND) return fail(WS_ERR_UNSUPPORTED, "unknown flags 0x%x", (unsigned)flags);
    if (!(scale > 0.f) || !std::isfinite(scale)) return fail(WS_ERR_UNSUPPORTED, "scale must be finite and > 0");
    if (num_q_heads % kv->num_kv_heads)
        return fail(WS_ERR_HEADS, "num_q_heads %d not a multiple of num_kv_heads %d", (int)num_q_heads,
                    (int)kv->num_kv_heads);
    if (lse && ((uintptr_t)lse & 3u)) return fail(WS_ERR_ALIGN, "lse must be 4-byte aligned");
    const bool fuse = (flags & WS_FUSE_APPEND) != 0;
    int64_t max_k = 0;
    for (int b = 0; b < batch; ++b) {
        if (cache_lens_host[b] < 0) return fail(WS_ERR_SHAPE, "cache_lens[%d] = %d", b, (int)cache_lens_host[b]);
        if (nl_host && (nl_host[b] < 1 || nl_host[b] > new_len))
            return fail(WS_ERR_SHAPE, "new_lens[%d] = %d outside [1, new_len %d]", b, (int)nl_host[b], (int)new_len);
        const int64_t nl = nl_host ? nl_host[b] : new_len;
        const int64_t need = (int64_t)cache_lens_host[b] + (fuse ? nl : 0);
        if (int rc = check_pages(kv, b, need)) return rc;
        if ((int64_t)cache_lens_host[b] + nl > max_k) max_k = (int64_t)cache_lens_host[b] + nl;
    }
    if (max_k > INT32_MAX) return fail(WS_ERR_SHAPE, "too many keys");
    if (text_host)
        for (int b = 0; b < batch; ++b)
            if (text_host[b] < 0 || text_host[b] > new_len)
                return fail(WS_ERR_OFFSETS, "text_starts[%d] = %d outside [0, new_len %d]", b, (int)text_host[b],
                            (int)new_len);
    if ((int64_t)(num_q_heads / kv->num_kv_heads) * new_len > WS_MAX_STEP_ROWS)
        return fail(WS_ERR_SHAPE, "new_len x query heads per KV head exceeds %lld", (long long)WS_MAX_STEP_ROWS);
    int cus = 0;
    if (int e = ws::current_device_cus(&cus))
        return fail(WS_ERR_HIP, "cannot query the device's compute units (hip error %d)", e);
    const StepPlan plan = plan_step(cus, batch, num_q_heads, kv->num_kv_heads, new_len, max_k, nl_host);
    const size_t need_ws = step_workspace(plan, batch, num_q_heads, kv->num_kv_heads, new_len);
    if (noalloc) {
        // the library's per-device scratch array stands in for the workspace
        if (need_ws > ws::NOALLOC_SCRATCH_BYTES)
            return fail(WS_ERR_WORKSPACE,
                        "this step needs %zu bytes of split partials; the allocation-free entry point "
                        "holds at most %zu (use ws_block_causal_attn_fwd with a workspace)",
                        need_ws, ws::NOALLOC_SCRATCH_BYTES);
        workspace = nullptr;
        workspace_bytes = 0;
        if (need_ws > 0) {
            if (int e = ws::scratch_address(&workspace))
                return fail(WS_ERR_HIP, "cannot look up the scratch array's device address (hip error %d)", e);
            workspace_bytes = ws::NOALLOC_SCRATCH_BYTES;
        }
    }
    if (need_ws > 0 && (!workspace || workspace_bytes < need_ws || !aligned16(workspace)))
        return fail(WS_ERR_WORKSPACE, "workspace needs %zu bytes (16-byte aligned), got %zu", need_ws,
                    workspace ? workspace_bytes : (size_t)0);

    ws::AttnArgs a{};
    a.q = (const uint16_t *)q.ptr; a.q_sb = q.stride_b; a.q_st = q.stride_t; a.q_sh = q.stride_h;
    a.kc = (const uint16_t *)k_new.ptr; a.kc_sb = k_new.stride_b; a.kc_st = k_new.stride_t; a.kc_sh = k_new.stride_h;
    a.vc = (const uint16_t *)v_new.ptr; a.vc_sb = v_new.stride_b; a.vc_st = v_new.stride_t; a.vc_sh = v_new.stride_h;
    a.kpool = (uint16_t *)kv->k_pool; a.vpool = (uint16_t *)kv->v_pool;
    a.page_table = kv->page_table_dev; a.max_pages = kv->max_pages_per_seq;
    a.cache_lens = cache_lens_dev;
    a.out = out.ptr; a.o_sb = out.stride_b; a.o_st = out.stride_t; a.o_sh = out.stride_h;
    a.out_f32 = out.dtype == WS_DTYPE_F32;
    a.lse = lse;
    a.B = batch; a.Lq = new_len; a.Hq = num_q_heads; a.Hkv = kv->num_kv_heads; a.G = num_q_heads / kv->num_kv_heads;
    a.mode = ws::MODE_STEP;
    a.fuse_append = fuse;
    a.nsplit = plan.nsplit;
    a.nqt = plan.nqt;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.gi = 1;
    a.nrows = a.G * new_len;
    a.nrb = (a.nrows + 31) / 32;
    if (plan.nsplit > 1) {
        a.part_o = (float *)workspace;
        a.part_ml = a.part_o + (size_t)plan.nsplit * batch * a.Hkv * a.nrb * 32 * kv->head_dim;
    }
    if (text_host) {
        a.text_starts = text_dev;
        a.has_text = 1;
    }
    if (nl_host) {
        a.new_lens = nl_dev;
        a.has_new_lens = 1;
    }
    if (batch <= ws::LENS_IN_ARGS) {
        a.lens_in_args = 1;
        for (int b = 0; b < batch; ++b) {
            a.lens_arg[b] = cache_lens_host[b];
            a.text_arg[b] = text_host ? text_host[b] : new_len;
            a.nl_arg[b] = nl_host ? nl_host[b] : new_len;
        }
    }
    if (!finish_work(a)) return fail(WS_ERR_SHAPE, "too many work items");
    if (int e = ws::launch_attention(a, kv->head_dim, plan.shape, stream))
        return fail(WS_ERR_HIP, "attention launch failed (hip error %d)", e);
    if (plan.nsplit > 1)
        if (int e = ws::launch_combine(a, kv->head_dim, stream))
            return fail(WS_ERR_HIP, "combine launch failed (hip error %d)", e);
    return ok();
}

// Whole-sequence prefill (text_* NULL: no token-causal segments).
int prefill_impl(ws_tensor4 q, ws_tensor4 k, ws_tensor4 v, const ws_paged_kv *kv_or_null,
                 const int32_t *block_offsets_host, const int32_t *block_offsets_dev,
                 const int32_t *text_host, const int32_t *text_dev,
                 int32_t batch, int32_t seq_len, int32_t num_blocks, int32_t num_q_heads,
                 int32_t num_kv_heads, int32_t head_dim, float scale, ws_tensor4 out,
                 float *lse, void *stream) {
    if (batch < 0 || seq_len < 0 || num_blocks < 0 || num_q_heads <= 0 || num_kv_heads <= 0)
        return fail(WS_ERR_SHAPE, "batch %d, seq_len %d, num_blocks %d, heads %d/%d", (int)batch, (int)seq_len,
                    (int)num_blocks, (int)num_q_heads, (int)num_kv_heads);
    if (batch == 0 || seq_len == 0) return ok();  // no token: nothing is read or written
    const bool paged = !k.ptr && !v.ptr;
    if (paged) {
        if (!kv_or_null) return fail(WS_ERR_NULL, "k/v are NULL and no paged cache was given");
        if (int rc = check_paged(kv_or_null)) return rc;
    } else {
        if (int rc = check_kv_tensor("k", k)) return rc;
        if (int rc = check_kv_tensor("v", v)) return rc;
    }
    if (int rc = check_tensor("q", q, false)) return rc;
    if (int rc = check_tensor("out", out, true)) return rc;
    if (!block_offsets_host || !block_offsets_dev) return fail(WS_ERR_NULL, "block offsets pointer is NULL");
    if (int rc = check_head_dim(head_dim)) return rc;
    if (!(scale > 0.f) || !std::isfinite(scale)) return fail(WS_ERR_UNSUPPORTED, "scale must be finite and > 0");
    if (num_q_heads % num_kv_heads)
        return fail(WS_ERR_HEADS, "num_q_heads %d not a multiple of num_kv_heads %d", (int)num_q_heads,
                    (int)num_kv_heads);
    if (paged && (kv_or_null->num_kv_heads != num_kv_heads || kv_or_null->head_dim != head_dim))
        return fail(WS_ERR_HEADS, "paged cache has %d KV heads of dim %d, call says %d of dim %d",
                    (int)kv_or_null->num_kv_heads, (int)kv_or_null->head_dim, (int)num_kv_heads, (int)head_dim);
    if (lse && ((uintptr_t)lse & 3u)) return fail(WS_ERR_ALIGN, "lse must be 4-byte aligned");
    for (int b = 0; b < batch; ++b) {
        const int32_t *off = block_offsets_host + (int64_t)b * (num_blocks + 1);
        if (off[0] != 0) return fail(WS_ERR_OFFSETS, "block_offsets[%d][0] = %d, must be 0", b, (int)off[0]);
        for (int n = 0; n < num_blocks; ++n) {
            if (off[n + 1] < off[n])
                return fail(WS_ERR_OFFSETS, "block_offsets[%d] decreases at %d", b, n + 1);
            if (text_host) {
                const int32_t t = text_host[(int64_t)b * num_blocks + n];
                if (t < off[n] || t > off[n + 1])
                    return fail(WS_ERR_OFFSETS, "text_starts[%d][%d] = %d outside block [%d, %d]", b, n, (int)t,
                                (int)off[n], (int)off[n + 1]);
            }
        }
        if (off[num_blocks] != seq_len)
            return fail(WS_ERR_OFFSETS, "block_offsets[%d][%d] = %d, must equal seq_len %d", b, (int)num_blocks,
                        (int)off[num_blocks], (int)seq_len);
        if (paged)
            if (int rc = check_pages(kv_or_null, b, seq_len)) return rc;
    }

    const ws::TileShape shape = plan_prefill(seq_len);
    ws::AttnArgs a{};
    a.q = (const uint16_t *)q.ptr; a.q_sb = q.stride_b; a.q_st = q.stride_t; a.q_sh = q.stride_h;
    if (paged) {
        a.kpool = (uint16_t *)kv_or_null->k_pool; a.vpool = (uint16_t *)kv_or_null->v_pool;
        a.page_table = kv_or_null->page_table_dev; a.max_pages = kv_or_null->max_pages_per_seq;
        a.paged = 1;
    } else {
        a.kc = (const uint16_t *)k.ptr; a.kc_sb = k.stride_b; a.kc_st = k.stride_t; a.kc_sh = k.stride_h;
        a.vc = (const uint16_t *)v.ptr; a.vc_sb = v.stride_b; a.vc_st = v.stride_t; a.vc_sh = v.stride_h;
    }
    a.offsets = block_offsets_dev;
    a.nb = num_blocks;
    if (text_host) {
        a.text_starts = text_dev;
        a.has_text = 1;
    }
    a.out = out.ptr; a.o_sb = out.stride_b; a.o_st = out.stride_t; a.o_sh = out.stride_h;
    a.out_f32 = out.dtype == WS_DTYPE_F32;
    a.lse = lse;
    a.B = batch; a.Lq = seq_len; a.Hq = num_q_heads; a.Hkv = num_kv_heads; a.G = num_q_heads / num_kv_heads;
    a.mode = ws::MODE_PREFILL;
    a.nsplit = 1;
    a.gi = a.G;
    a.nrows = seq_len;
    a.nqt = (seq_len + shape.qtile() - 1) / shape.qtile();
    a.scale_log2 = scale * 1.4426950408889634f;
    if (!finish_work(a)) return fail(WS_ERR_SHAPE, "too many work items");
    if (int e = ws::launch_attention(a, head_dim, shape, stream))
        return fail(WS_ERR_HIP, "prefill launch failed (hip error %d)", e);
    return ok();
}

}  // namespace
