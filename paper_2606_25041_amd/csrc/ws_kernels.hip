// gfx950 (MI355X) kernels for block-causal streaming attention.
//
// Block-causal rule (Wan-Streamer v0.1, Abstract; Sec. 1 with Fig. 1): a
// token sees its whole own block and every earlier block; a block may end in
// a token-causal segment (the thinker's language and state slots, Sec. 1 and
// Sec. 2.4) whose tokens see the segment only up to themselves.  The step
// kernel runs the current unit against its full-history cache (Sec. 2.4);
// the prefill kernel covers whole sequences (Sec. 2.4, system prefill); the
// append kernel commits a KV slice to the paged cache (Sec. 2.4).  The
// gradient kernels, which serve training in the same causal format
// (Sec. 2.3), are in ws_bwd.hip.
//
// Attention kernel design (one work-group = one work item: a tile of 256
// query rows of one (stream, KV head) group and one KV split, 8 waves x 32
// rows; in the prefill the rows are tokens of one query head of the group,
// in a step they are packed (token, query head) rows, every query head of
// the group for consecutive new tokens):
//  * S^T = K Q^T on v_mfma_f32_32x32x16_bf16: K (A operand) from LDS, Q (B
//    operand) resident in registers.  In the 32x32 accumulator layout a lane
//    owns one query column and 16 keys, so row max/sum are in-lane plus one
//    v_permlane32_swap per 64-key tile.
//  * Online softmax in the log2 domain (scale*log2(e) folded into one FMA),
//    fp32 running max/sum per lane, lazy rescale of O; a tile's max is only
//    taken when some row may need a larger running max.
//  * O^T += V^T P^T on the same MFMA: P stays in registers (the accumulator
//    layout of S^T is exactly the B-operand layout once the 16 keys of each
//    MFMA step are permuted consistently on both operands); V is read with
//    ds_read_b64_tr_b16 from a row-major LDS tile, so no transpose pass.
//  * K/V tiles of 64 keys (= one cache page) go from global memory straight
//    into a 5-stage LDS ring (global_load_lds_dwordx4), three tiles in flight
//    while the current one is used; rows are XOR-swizzled in 16-byte chunks
//    so both the K reads and the V transpose reads are bank-conflict free.
//  * Two waves share each SIMD and run the same loop one block apart: while
//    one issues the MFMAs of a tile (S^T of this one, P V of the previous
//    tile), the other computes its softmax; a work-group barrier separates
//    the blocks.
//  * Tiles past the last visible key of the query tile are never loaded
//    (block-granularity skip); tiles fully visible to every row of the query
//    tile run without element masks; only the tiles straddling a block
//    boundary (or the end of the keys) apply per-element masks.
//  * Work items are ordered by KV group (stream, KV head) and mapped
//    XCD-aware: consecutive logical items land on the same XCD so query heads
//    and query tiles that read the same K/V share that XCD's L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ws_kernels.h"
#include "ws_device_util.h"

namespace ws {
namespace {

constexpr int KT = 64;        // keys per tile (= page size)
constexpr float RESCALE_LOG2 = 8.f;  // lazy-rescale threshold (log2 units)
constexpr float RESCALE_BOUND = 256.f;  // 2^RESCALE_LOG2
constexpr int NSTAGE = 5;            // K/V tiles resident in the LDS ring (loads three tiles ahead)
constexpr int RAHEAD = 4;            // LDS operand reads issued this many MFMAs ahead

// The fused append's share of step work item ai (of nqt * nsplit per
// (stream, KV head)): the group's items split the new tokens evenly; tokens
// t >= nl are padding and not committed.  One 16-byte chunk per thread.
template <int D, int NT>
__device__ __forceinline__ void append_share(const AttnArgs &a, int b, int kvh, int ai, int n_pool, int nl,
                                             const int32_t *ptab, int tid) {
    constexpr int CH = D / 8;
    const int napp = a.nqt * a.nsplit;
    const int s0 = (int)((int64_t)ai * a.Lq / napp);
    const int n = max(min((int)((int64_t)(ai + 1) * a.Lq / napp), nl) - s0, 0) * CH;
    for (int u = tid; u < n; u += NT) {
        const int t = s0 + u / CH, c = u % CH;
        const int pos = n_pool + t;
        const int64_t dst = (((int64_t)ptab[pos >> 6] * a.Hkv + kvh) * KT + (pos & 63)) * D + 8 * c;
        *(u32x4 *)(a.kpool + dst) = *(const u32x4 *)(a.kc + b * a.kc_sb + (int64_t)t * a.kc_st + kvh * a.kc_sh + 8 * c);
        *(u32x4 *)(a.vpool + dst) = *(const u32x4 *)(a.vc + b * a.vc_sb + (int64_t)t * a.vc_st + kvh * a.vc_sh + 8 * c);
    }
}

template <int D, int NW, int NB>
__global__ __launch_bounds__(NW * 64) void attn_kernel(const AttnArgs a) {
    constexpr int NT = NW * 64;
    constexpr int QT = NW * 32 * NB;       // query rows per work-group
    constexpr int ROWB = 2 * D;            // bytes of one key row
    constexpr int TILEB = KT * ROWB;       // bytes of one K (or V) tile
    constexpr int RPW = 1024 / ROWB;       // key rows per wave-wide 16-byte load
    constexpr int LPR = ROWB / 16;         // lanes per key row in such a load
    constexpr int NWD = NW / 2;            // waves that load tiles (the leading half)
    constexpr int NI = TILEB / (NWD * 1024);  // wave-wide loads per loading wave per tile, each of K and V
    constexpr int KK = D / 16;             // MFMA k-steps over head_dim for S^T
    constexpr int MD = D / 32;             // 32-row blocks of head_dim for O^T
    constexpr int VRING = NSTAGE * TILEB;  // byte offset of the V ring
    static_assert(NI >= 1 && TILEB % (NWD * 1024) == 0, "a tile splits into wave-wide loads");
    __shared__ __attribute__((aligned(1024))) char smem[2 * NSTAGE * TILEB];

    // ---- work item ------------------------------------------------------
    // The launch parameters the decode and the query loads need are read in
    // one batch (the asm makes them all live at once, so the compiler issues
    // their loads together and waits once, instead of one round trip per
    // field as each is first used); divisions use the host's dividers.
    const uint32_t bid = blockIdx.x;
    uint32_t per_xcd = a.per_xcd, n_work = a.n_work, per_group = a.per_group, per_qt = a.per_qt;
    uint32_t G = a.G, gi = a.gi, Hkv = a.Hkv, mode = a.mode, nqt = a.nqt, nrows = a.nrows, lens0 = a.lens_arg[0];
    uint32_t has_nl = a.has_new_lens;
    FastDiv fd_group = a.fd_group, fd_qt = a.fd_qt, fd_g = a.fd_g, fd_hkv = a.fd_hkv, fd_split = a.fd_split;
    FastDiv fd_gq = a.fd_gq;
    const uint16_t *qptr = a.q;
    int64_t q_sb = a.q_sb, q_st = a.q_st, q_sh = a.q_sh;
    asm volatile("" : "+s"(per_xcd), "+s"(n_work), "+s"(per_group), "+s"(per_qt), "+s"(G), "+s"(gi), "+s"(Hkv),
                      "+s"(mode), "+s"(nqt), "+s"(nrows), "+s"(lens0), "+s"(fd_group.mul), "+s"(fd_group.shift),
                      "+s"(fd_qt.mul), "+s"(fd_qt.shift), "+s"(fd_g.mul), "+s"(fd_g.shift), "+s"(fd_hkv.mul),
                      "+s"(fd_hkv.shift), "+s"(fd_split.mul), "+s"(fd_split.shift), "+s"(fd_gq.mul),
                      "+s"(fd_gq.shift), "+s"(qptr), "+s"(q_sb), "+s"(q_st), "+s"(q_sh), "+s"(has_nl));
    const uint32_t w = (bid % NUM_XCD) * per_xcd + bid / NUM_XCD;
    if (w >= n_work) return;
    const uint32_t group = fastdiv(w, fd_group);
    const uint32_t idx = w - group * per_group;
    const uint32_t qi = fastdiv(idx, fd_qt);
    const uint32_t rem = idx - qi * per_qt;
    const uint32_t split = fastdiv(rem, fd_g);
    const int hh = (int)(rem - split * gi);
    // Groups are taken stream-major; a step over blocks of different lengths
    // takes them KV-head-major instead, so that the contiguous range of items
    // each XCD runs mixes long and short streams rather than holding a few
    // streams only.
    int b, kvh;
    if (has_nl) {
        kvh = (int)fastdiv(group, a.fd_b);
        b = (int)(group - (uint32_t)kvh * (uint32_t)a.B);
    } else {
        b = (int)fastdiv(group, fd_hkv);
        kvh = (int)(group - b * Hkv);
    }
    const int hq = kvh * (int)G + hh;   // (prefill; a step's rows span the group's heads)
    const bool step = mode == MODE_STEP;
    // token and query head of packed row p (see AttnArgs)
    auto row_token = [&](int p) -> int { return step ? (int)fastdiv((uint32_t)p, fd_gq) : p; };
    auto row_head = [&](int p, int t) -> int { return step ? kvh * (int)G + (p - t * (int)G) : hq; };
    const int qt = step ? (int)qi : (int)(nqt - 1 - qi);  // prefill: heaviest tiles first
    const int q0 = qt * QT;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int hf = lane >> 5;     // which half of the wave
    const int l32 = lane & 31;
    // 32-row block of the tile this wave computes: the trailing waves (which
    // issue no tile loads) take the first blocks, so a small block's rows go
    // to waves without load duty
    const int rblk = (wave + NW / 2) % NW;

    // A step tile whose first token lies past its stream's new block (blocks
    // of different lengths, padded) holds no real row: it computes nothing
    // and leaves its rows' outputs unwritten, but still does its share of
    // the fused append.  Decided before any load is issued.
    if (step && has_nl) {
        const int nl0 = a.lens_in_args ? a.nl_arg[b] : ld_uniform(a.new_lens, b);
        if ((int)fastdiv((uint32_t)q0, fd_gq) >= nl0) {
            if (a.fuse_append) {
                const int np0 = a.lens_in_args ? a.lens_arg[b] : ld_uniform(a.cache_lens, b);
                append_share<D, NT>(a, b, kvh, (int)(qi * a.nsplit + split), np0, nl0,
                                    a.page_table + (int64_t)b * a.max_pages, tid);
            }
            return;
        }
    }

    // Query rows of this wave go global -> LDS -> registers, issued first
    // thing: the direct loads stay in order with the tile loads, so one
    // counted wait covers both.  They are staged in the last two ring stages
    // (of the K ring for waves 0..3, of the V ring for waves 4..7), which are
    // first refilled in loop steps t_begin and t_begin + 1, after every wave
    // has passed the prologue barrier.  The layout is that of a key tile, so the fragments
    // are read like K.
    static_assert(NB == 1, "query staging holds 32 rows per wave");
    constexpr int QI = 32 * ROWB / 1024;   // wave-wide loads per wave
    const uint32_t q_stage = (uint32_t)((wave < 4 ? 0 : VRING) + (NSTAGE - 2) * TILEB + (wave & 3) * 32 * ROWB);
    {
        const char *qg = (const char *)(qptr + b * q_sb);
#pragma unroll
        for (int i = 0; i < QI; ++i) {
            const int r = i * RPW + lane / LPR;   // row within the wave's 32
            const int ch = (lane % LPR) ^ swz<D>(r);
            const int p = min(q0 + rblk * 32 + r, (int)nrows - 1);
            const int t = row_token(p);
            const int h = row_head(p, t);
            dma16(qg + (int64_t)t * (2 * q_st) + (int64_t)h * (2 * q_sh) + 16 * ch, lds_addr(smem) + q_stage + i * 1024);
        }
    }

    // ---- key range ------------------------------------------------------
    // Every row sees a prefix [0, kend) of the keys, and kend does not
    // decrease along the rows of a tile, so the tile's first and last rows
    // give the keys all rows see (kfull) and the keys any row sees (k_hi).
    const int32_t *offs = step ? nullptr : a.offsets + (int64_t)b * (a.nb + 1);
    const int32_t *text = (!step && a.has_text) ? a.text_starts + (int64_t)b * a.nb : nullptr;
    int n_pool, k_hi, kfull, ts = 0, nl = 0;
    if (step) {
        n_pool = !a.lens_in_args ? ld_uniform(a.cache_lens, b) : b == 0 ? (int)lens0 : a.lens_arg[b];
        // start of the new block's token-causal segment (Lq: none) and the
        // block's length (Lq: no padding); new token t sees
        // n_pool + min(nl, max(ts, t + 1)) keys
        ts = a.lens_in_args ? a.text_arg[b] : a.has_text ? ld_uniform(a.text_starts, b) : a.Lq;
        nl = a.lens_in_args ? a.nl_arg[b] : a.has_new_lens ? ld_uniform(a.new_lens, b) : a.Lq;
        const int t_last = (int)fastdiv((uint32_t)(min(q0 + QT, (int)nrows) - 1), fd_gq);
        k_hi = n_pool + min(nl, max(ts, t_last + 1));
        kfull = n_pool + min(nl, max(ts, (int)fastdiv((uint32_t)q0, fd_gq) + 1));
    } else {
        n_pool = a.paged ? a.Lq : 0;
        const int q_last = min(q0 + QT, a.Lq) - 1;
        k_hi = row_key_end<true>(offs, text, a.nb, q_last);
        kfull = row_key_end<true>(offs, text, a.nb, q0);
    }
    const int ntile = (k_hi + KT - 1) / KT;
    // (split * ntile < 2^31: ntile < 2^25 and split < MAX_SPLITS = 32)
    const int t_begin = (int)fastdiv(split * (uint32_t)ntile, fd_split);
    const int t_end = (int)fastdiv((split + 1) * (uint32_t)ntile, fd_split);

    // ---- page ids -------------------------------------------------------
    // The first four tiles' pages are read up front; later ones one loop
    // step before their tile's loads are issued (a scalar load, waited for
    // with the tile loads), so no page-table read sits in front of them.
    const int32_t *ptab = a.page_table + (int64_t)b * a.max_pages;
    const int tp_end = min(t_end, (n_pool + KT - 1) / KT);   // tiles with cache rows
    auto page_glb = [&](int t) -> int { return t < tp_end ? ld_uniform(ptab, t) : 0; };

    // ---- this lane's query rows -------------------------------------------
    // row n of the lane: q0 + rblk * 32 * NB + 32 * n + l32 (the fragments
    // are staged through LDS in the pipeline prologue, below)
    int row[NB], kend[NB], tok[NB], hqr[NB];
    bf16x8 qf[NB][KK];
#pragma unroll
    for (int n = 0; n < NB; ++n) {
        row[n] = q0 + rblk * 32 * NB + 32 * n + l32;
        const int pc = min(row[n], (int)nrows - 1);
        tok[n] = row_token(pc);
        hqr[n] = row_head(pc, tok[n]);
        kend[n] = step ? n_pool + min(nl, max(ts, tok[n] + 1)) : row_key_end<false>(offs, text, a.nb, tok[n]);
    }

    // ---- direct-to-LDS tile loads -----------------------------------------
    // The leading waves (wave < NWD) load the tiles.  Wave-wide load i of
    // such a wave fills tile bytes [(i * NWD + wave) * 1024, +1024): lane
    // `lane` writes 16 bytes at +16 * lane, i.e. slot lane % LPR of key row
    // lrow0 + i * NWD * RPW, and so fetches the chunk that belongs there,
    // lch = slot ^ swz(row).  The swizzle depends on the row modulo 16 only,
    // so lch is the same for all i.
    static_assert((NWD * RPW) % 16 == 0, "the swizzle must repeat across a wave's loads");
    const int lrow0 = wave * RPW + lane / LPR;
    const int lch = (lane % LPR) ^ swz<D>(lrow0);
    const char *kpool_b = (const char *)a.kpool;
    const char *vpool_b = (const char *)a.vpool;
    const char *kc_b = (const char *)(a.kc + b * a.kc_sb + kvh * a.kc_sh);
    const char *vc_b = (const char *)(a.vc + b * a.vc_sb + kvh * a.vc_sh);
    const int64_t kst2 = 2 * a.kc_st, vst2 = 2 * a.vc_st;
    // per-lane byte offsets: within a (page, KV head) tile, and within the
    // contiguous rows starting at this wave's first row (token strides are
    // below 2^24 elements, checked on the host)
    uint32_t lofs_p = (uint32_t)(lrow0 * ROWB + 16 * lch);
    uint32_t lofs_k = (uint32_t)((lane / LPR) * kst2 + 16 * lch);
    uint32_t lofs_v = (uint32_t)((lane / LPR) * vst2 + 16 * lch);
    // Loads of one tile u (its physical page, if cached, is `page`,
    // wave-uniform) into ring stage s: NI wave-wide loads for K and for V.
    // A tile inside one cache page or inside the contiguous keys is loaded
    // from a wave-uniform base + i * step and a per-lane offset, so its loads
    // can be spread out (issue_part); a tile straddling the cache end or the
    // last key is loaded at once with per-lane addresses (issue_straddle).
    struct TileLoad {
        const char *bk, *bv;   // wave-uniform bases of load 0
        int64_t sk, sv;        // base step per load
        uint32_t ok, ov;       // per-lane byte offsets
        uint32_t kd, vd;       // LDS destination of load 0 of this wave
        bool straddle;
    };
    auto plan_tile = [&](int u, int s, int page) -> TileLoad {
        const int kt = u * KT;
        TileLoad t;
        t.kd = lds_addr(smem) + s * TILEB + wave * 1024;
        t.vd = t.kd + VRING;
        t.straddle = false;
        if (kt + KT <= n_pool) {
            // whole tile in one cache page
            const int64_t tb = ((int64_t)page * a.Hkv + kvh) * TILEB;
            t.bk = kpool_b + tb;
            t.bv = vpool_b + tb;
            t.sk = t.sv = NWD * 1024;
            t.ok = t.ov = lofs_p;
        } else if (kt >= n_pool && kt + KT <= k_hi) {
            // whole tile in the contiguous keys
            const int64_t j0 = kt - n_pool + wave * RPW;
            t.bk = kc_b + j0 * kst2;
            t.bv = vc_b + j0 * vst2;
            t.sk = NWD * RPW * kst2;
            t.sv = NWD * RPW * vst2;
            t.ok = lofs_k;
            t.ov = lofs_v;
        } else {
            t.straddle = true;
        }
        return t;
    };
    auto issue_part = [&](const TileLoad &t, int i) {
        dma16s(t.bk + i * t.sk, t.ok, t.kd + i * NWD * 1024);
        dma16s(t.bv + i * t.sv, t.ov, t.vd + i * NWD * 1024);
    };
    // rows past the end repeat the last key (their scores are masked)
    auto issue_straddle = [&](int u, int s, int page) {
        const int kt = u * KT;
        const uint32_t kd = lds_addr(smem) + s * TILEB + wave * 1024;
        const uint32_t vd = kd + VRING;
        const int64_t tb = ((int64_t)page * a.Hkv + kvh) * TILEB;
        const char *kg = kpool_b + tb, *vg = vpool_b + tb;
        const int64_t c0 = (int64_t)(kt - n_pool);   // contiguous row of the tile's first key
        const char *kcg = kc_b + c0 * kst2, *vcg = vc_b + c0 * vst2;
        const uint32_t lofs_c = lofs_p - lrow0 * ROWB;   // the chunk's byte offset in a row
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int r = min(lrow0 + i * NWD * RPW, k_hi - 1 - kt);   // row within the tile
            const char *gk, *gv;
            if (kt + r < n_pool) {
                gk = kg + (uint32_t)(r * ROWB) + lofs_c;
                gv = vg + (uint32_t)(r * ROWB) + lofs_c;
            } else {
                gk = kcg + (uint32_t)(r * kst2) + lofs_c;
                gv = vcg + (uint32_t)(r * vst2) + lofs_c;
            }
            dma16(gk, kd + i * NWD * 1024);
            dma16(gv, vd + i * NWD * 1024);
        }
    };
    // all loads of tile u at once
    auto issue_tile = [&](int u, int s, int page) {
        const TileLoad t = plan_tile(u, s, page);
        if (t.straddle) {
            issue_straddle(u, s, page);
        } else {
#pragma unroll
            for (int i = 0; i < NI; ++i) issue_part(t, i);
        }
        // the waits count this tile's loads as one group: keep later memory
        // operations from being moved in between
        asm volatile("" ::: "memory");
    };
    // wait until at most `younger` tiles' loads are still in flight
    auto wait_tiles = [&](int younger) {
        if (younger >= 2) wait_vm_lgkm<4 * NI>();
        else if (younger == 1) wait_vm_lgkm<2 * NI>();
        else wait_vm_lgkm<0>();
    };

    // ---- LDS read addresses -----------------------------------------------
    // K (A operand of S^T = K Q^T): lane (l32, hf) reads key row 32 * mb + l32,
    // chunk 2 * kk + hf, at kbase ^ (32 * kk): the row offset has no bits
    // below 128 and chunk 2 * kk ^ swz only changes bits 5.. of the slot.
    uint32_t kbase = l32 * ROWB + 16 * (hf ^ swz<D>(l32));
    // V^T fragments (A operand of O^T += V^T P^T) by transpose reads: lane
    // reads key rows 16 * ks4 + vr and +8, 4 head-dim columns of chunk
    // 4 * md + vc, at vbase[e] ^ (64 * md).
    const int j16 = lane & 15;
    uint32_t vbase[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const int vr = 4 * hf + (j16 >> 2) + 8 * e;
        const int vc = 2 * ((lane >> 4) & 1) + ((j16 & 3) >> 1);
        vbase[e] = VRING + vr * ROWB + 16 * (vc ^ swz<D>(vr)) + 8 * (j16 & 1);
    }

    auto read_q = [&]() {
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            qf[0][kk] = *(const bf16x8 *)(smem + q_stage + (kbase ^ (32 * kk)));
    };

    const float c2 = a.scale_log2;
    f32x16 o[NB][MD];
    float m[NB], l[NB];
#pragma unroll
    for (int n = 0; n < NB; ++n) {
        m[n] = -INFINITY;
        l[n] = 0.f;
#pragma unroll
        for (int md = 0; md < MD; ++md)
#pragma unroll
            for (int v = 0; v < 16; ++v) o[n][md][v] = 0.f;
    }

    constexpr int NQK = 2 * KK;       // K fragments (steps) of S^T per tile; NB MFMAs each
    constexpr int NPV = 4 * MD;       // V fragments (steps) of O^T per tile; NB MFMAs each
    constexpr int SPQ = 32 * NB / NQK;   // softmax scores per S^T step
    constexpr int SPV = 32 * NB / NPV;   // scores per O^T step folded into the next row max
    static_assert(SPQ % 2 == 0 && SPV % 2 == 0, "scores go in pairs");
    typedef f32x16 Tile[NB][2];      // S^T of one tile: per query block, two 32-key blocks

    // (soff: byte offset of a ring stage, a multiple of TILEB, so adding it
    // commutes with the XORs on the low address bits)
    // K fragment of S^T step i (kk = i / 2, key block mb = i % 2)
    auto kread = [&](uint32_t kb, int i) -> bf16x8 {
        return *(const bf16x8 *)(smem + (i & 1) * 32 * ROWB + (kb ^ (32 * (i >> 1))));
    };
    // V^T fragment of O^T step i (ks4 = i / MD, md = i % MD) by two
    // transpose reads
    auto vread = [&](uint32_t v0, uint32_t v1, int i) -> bf16x8 {
        const int ks4 = i / MD, md = i % MD;
        const i16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_i16x4 *)(smem + ks4 * 16 * ROWB + (v0 ^ (64 * md))));
        const i16x4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_i16x4 *)(smem + ks4 * 16 * ROWB + (v1 ^ (64 * md))));
        // whole-vector reinterpretation: element-wise bf16 casts of the
        // transpose-read result were lowered to a splat
        return __builtin_bit_cast(bf16x8, __builtin_shufflevector(va, vb, 0, 1, 2, 3, 4, 5, 6, 7));
    };
    // score e (0..32*NB-1) of a tile: query block n = e / 32, and within it
    // in P's B-operand order (fragment ks4 = e % 32 / 8 holds keys
    // 8 * (ks4 & 1) + e % 8 of key block ks4 / 2)
    auto score = [&](const Tile &sc, int e) -> float { return sc[e >> 5][(e >> 4) & 1][e & 15]; };
    // P weights of a tile: 2^(s * c2 - m), rounded to bf16 for P.V, and their
    // fp32 lane sums ls (so lse is exact to fp32 rounding).  One straight block:
    // all exponents, then all exps, then the packs and a pairwise sum, so
    // the dependent steps of different scores overlap.
    auto softmax_weights = [&](const Tile &sc, bf16x8 (&pf)[NB][4], const float (&m_use)[NB], float (&ls)[NB]) {
#pragma unroll
        for (int n = 0; n < NB; ++n) {
            float x[32];
#pragma unroll
            for (int f = 0; f < 32; ++f) x[f] = __builtin_fmaf(score(sc, 32 * n + f), c2, -m_use[n]);
#pragma unroll
            for (int f = 0; f < 32; ++f) x[f] = fast_exp2(x[f]);
#pragma unroll
            for (int f = 0; f < 32; ++f) pf[n][f >> 3][f & 7] = (__bf16)x[f];
            // pairwise sum in a fixed order (the same for every tile)
#pragma unroll
            for (int w = 1; w < 32; w *= 2)
#pragma unroll
                for (int f = 0; f < 32; f += 2 * w) x[f] += x[f + w];
            ls[n] = x[0];
        }
    };
    // in-lane max of a tile's scores per query block; the other half-wave's
    // keys are folded in by update_max
    auto lane_max = [&](const Tile &sc, float (&mx)[NB]) {
#pragma unroll
        for (int n = 0; n < NB; ++n) {
            mx[n] = -INFINITY;
#pragma unroll
            for (int e = 0; e < 32; ++e) mx[n] = fmaxf(mx[n], score(sc, 32 * n + e));
        }
    };
    // element masks only where the tile is not visible to every row
    auto mask = [&](int t, Tile &sc) {
        const int kt = t * KT;
#pragma unroll
        for (int n = 0; n < NB; ++n)
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int key = kt + mb * 32 + (v >> 2) * 8 + 4 * hf + (v & 3);
                    if (key >= kend[n]) sc[n][mb][v] = -INFINITY;
                }
    };
    // Running max (log2 domain) from a tile's in-lane max, with lazy rescale:
    // m only moves when the tile max exceeds it by more than 2^RESCALE_LOG2,
    // so most tiles skip rescaling O and l (a wave-uniform branch).  Weights
    // stay <= 2^RESCALE_LOG2; O and l share the same m, so the quotient is
    // exact.
    auto update_max = [&](const float (&mx_lane)[NB]) {
#pragma unroll
        for (int n = 0; n < NB; ++n) {
            const float mx = halves_max(mx_lane[n]) * c2;
            const bool grow = mx > m[n] + RESCALE_LOG2;
            if (__builtin_amdgcn_ballot_w64(grow)) {
                // lanes that keep m scale by 1 (also while m is still -inf:
                // a row that sees no key of this tile); 0 from -inf
                const float m_new = grow ? mx : m[n];
                const float alpha = grow ? fast_exp2(m[n] - m_new) : 1.f;
                m[n] = m_new;
                l[n] *= alpha;
#pragma unroll
                for (int md = 0; md < MD; ++md)
#pragma unroll
                    for (int v = 0; v < 16; ++v) o[n][md][v] *= alpha;
            }
        }
    };
    auto max_shift = [&](float (&m_use)[NB]) {
#pragma unroll
        for (int n = 0; n < NB; ++n) m_use[n] = (m[n] == -INFINITY) ? 0.f : m[n];
    };
    // S^T[key][query] = K Q^T for the 64 keys of a stage x this wave's
    // 32 * NB queries.  Each step is fenced so the reads stay RAHEAD steps
    // ahead of their MFMAs.
    auto qk = [&](uint32_t soff, Tile &sn) {
        const uint32_t kb = kbase + soff;
#pragma unroll
        for (int n = 0; n < NB; ++n)
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int v = 0; v < 16; ++v) sn[n][mb][v] = 0.f;
        bf16x8 kf[RAHEAD + 1];
#pragma unroll
        for (int i = 0; i < RAHEAD; ++i) kf[i] = kread(kb, i);
#pragma unroll
        for (int i = 0; i < NQK; ++i) {
            if (i + RAHEAD < NQK) kf[(i + RAHEAD) % (RAHEAD + 1)] = kread(kb, i + RAHEAD);
#pragma unroll
            for (int n = 0; n < NB; ++n)
                sn[n][i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[i % (RAHEAD + 1)], qf[n][i >> 1], sn[n][i & 1], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // softmax of a tile: mask, running max, P weights and their sum
    auto softmax = [&](int t, Tile &sc, bf16x8 (&pf)[NB][4]) {
        if ((t + 1) * KT > kfull) {
            // (a real branch: the compiler would otherwise turn this rare
            // path into selects executed on every tile)
            asm volatile("" ::: "memory");
            mask(t, sc);
        }
        // Weights at the running max as it stands; the tile's max is only
        // taken when some row may need a larger one: a row that has seen no
        // key yet, or whose lane sum of weights exceeds 2^RESCALE_LOG2 (a
        // necessary condition for a score above m + RESCALE_LOG2; inf and
        // NaN land here too).  That path is the lazy-rescale update and the
        // weights again, so every weight stays <= 2^RESCALE_LOG2 either way.
        float m_use[NB], ls[NB];
        max_shift(m_use);
        softmax_weights(sc, pf, m_use, ls);
        bool slow = false;
#pragma unroll
        for (int n = 0; n < NB; ++n) slow = slow || m[n] == -INFINITY || !(ls[n] <= RESCALE_BOUND);
        if (__builtin_amdgcn_ballot_w64(slow)) {
            float mx[NB];
            lane_max(sc, mx);
            update_max(mx);
            max_shift(m_use);
            softmax_weights(sc, pf, m_use, ls);
        }
#pragma unroll
        for (int n = 0; n < NB; ++n) l[n] += ls[n];
    };
    // O^T[d][query] += V^T P^T from the V tile of a stage; V reads RAHEAD
    // steps ahead of their MFMAs
    auto pv = [&](uint32_t soff, const bf16x8 (&pf)[NB][4]) {
        const uint32_t v0 = vbase[0] + soff, v1 = vbase[1] + soff;
        bf16x8 vf[RAHEAD + 1];
#pragma unroll
        for (int i = 0; i < RAHEAD; ++i) vf[i] = vread(v0, v1, i);
#pragma unroll
        for (int i = 0; i < NPV; ++i) {
            if (i + RAHEAD < NPV) vf[(i + RAHEAD) % (RAHEAD + 1)] = vread(v0, v1, i + RAHEAD);
#pragma unroll
            for (int n = 0; n < NB; ++n)
                o[n][i % MD] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[i % (RAHEAD + 1)], pf[n][i / MD], o[n][i % MD], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // ---- pipeline ---------------------------------------------------------
    // Tile t lives in ring stage (t - t_begin) % NSTAGE.  Every wave runs
    // the same loop: step j is an MFMA block (S^T of tile j, then O += P V
    // of tile j-1), a work-group barrier, the VALU block (softmax of tile j)
    // and another barrier.  The second wave on each SIMD (waves NWD..NW-1,
    // SIMD = wave % 4) enters the loop one barrier late, so on every SIMD one
    // wave's softmax overlaps the other wave's MFMAs.  The leading waves
    // issue the loads of tile j+3 at the start of step j and wait for tile
    // j+1 before its last barrier: a stage is refilled only after the
    // trailing waves' last read of its tile, and its loads have three steps
    // to land.
    static_assert(NW == 8, "two waves per SIMD");
    const bool lead = wave < NWD;
    // a wave whose 32 rows all lie past the last row (a small block's tile)
    // only takes part in the loads and barriers
    const bool busy = q0 + rblk * 32 < (int)nrows;
    Tile S;
    bf16x8 pf[NB][4];
    const int n_tiles = t_end - t_begin;
    auto stage_off = [&](int t) -> uint32_t { return (uint32_t)((t - t_begin) % NSTAGE) * TILEB; };
    if (n_tiles > 0) {
        // Prologue: the leading waves issue the first three tiles and wait
        // for the first and their query rows (the other two stay in flight
        // into loop step t_begin, as in the steady state); the trailing
        // waves wait for their query rows.  The page-id reads are the only
        // loads the compiler sees here, so its own waits never cover the
        // tile loads.
        int pg_next = 0;   // page of tile j+3, read one step ahead
        if (lead) {
            const int pg0 = page_glb(t_begin), pg1 = page_glb(t_begin + 1), pg2 = page_glb(t_begin + 2);
            pg_next = page_glb(t_begin + 3);
            issue_tile(t_begin, 0, pg0);
            if (n_tiles > 1) issue_tile(t_begin + 1, 1, pg1);
            if (n_tiles > 2) issue_tile(t_begin + 2, 2, pg2);
            wait_tiles(min(2, n_tiles - 1));
        } else {
            wait_vm_lgkm<0>();
        }
        read_q();
        wait_vm_lgkm<63>();   // (LDS reads and writes complete; no vector-memory wait)
        wg_barrier();
        if (!lead) wg_barrier();
        for (int j = t_begin; j <= t_end; ++j) {
            // Addresses derived from these per-lane bases are cheap to
            // recompute; hidden from the optimiser here so that it does not
            // hoist them out of the loop and hold them in registers the
            // pipeline needs.
            asm volatile("" : "+v"(kbase), "+v"(vbase[0]), "+v"(vbase[1]), "+v"(lofs_p), "+v"(lofs_k), "+v"(lofs_v));
            if (busy) {
                // S^T of tile j first: its accumulators are complete long
                // before the softmax reads them after the barrier
                if (j < t_end) qk(stage_off(j), S);
                if (j > t_begin) pv(stage_off(j - 1), pf);
            }
            wg_barrier();
            // the leading waves issue the loads of tile j+3 here, ahead of
            // their softmax, rather than ahead of their MFMA block
            if (lead && j + 3 < t_end) issue_tile(j + 3, (j + 3 - t_begin) % NSTAGE, pg_next);
            if (busy && j < t_end) softmax(j, S, pf);
            // (read here, under the wait below: a scalar read left in flight
            // across the MFMA block would force full LDS drains there)
            if (lead && j + 4 < t_end) pg_next = page_glb(j + 4);
            // tile j+1 landed; tiles j+2 and j+3 may stay in flight
            if (lead && j + 1 < t_end) wait_tiles(min(2, t_end - 2 - j));
            wg_barrier();
        }
        if (lead) wg_barrier();
    } else {
        wait_vm_lgkm<0>();   // (the query loads)
    }

    // ---- epilogue -----------------------------------------------------------
#pragma unroll
    for (int n = 0; n < NB; ++n) {
        const float lt = halves_sum(l[n]);
        const int r = row[n];
        if (r >= (int)nrows) continue;
        const int t = tok[n], h = hqr[n];
        if (a.nsplit == 1) {
            const float inv = lt > 0.f ? 1.f / lt : 0.f;
            if (a.out_f32) {
                float *op = (float *)a.out + b * a.o_sb + (int64_t)t * a.o_st + h * a.o_sh;
#pragma unroll
                for (int md = 0; md < MD; ++md)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        f32x4 val;
#pragma unroll
                        for (int e = 0; e < 4; ++e) val[e] = o[n][md][4 * g + e] * inv;
                        *(f32x4 *)(op + 32 * md + 8 * g + 4 * hf) = val;
                    }
            } else {
                uint16_t *op = (uint16_t *)a.out + b * a.o_sb + (int64_t)t * a.o_st + h * a.o_sh;
#pragma unroll
                for (int md = 0; md < MD; ++md)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        u32x2 val;
                        val[0] = pack_bf16x2(o[n][md][4 * g + 0] * inv, o[n][md][4 * g + 1] * inv);
                        val[1] = pack_bf16x2(o[n][md][4 * g + 2] * inv, o[n][md][4 * g + 3] * inv);
                        *(u32x2 *)(op + 32 * md + 8 * g + 4 * hf) = val;
                    }
            }
            if (a.lse && hf == 0)
                a.lse[((int64_t)b * a.Hq + h) * a.Lq + t] = (m[n] + __builtin_amdgcn_logf(lt)) * 0.69314718055994531f;
        } else if (!a.out_f32) {
            // bf16 output: o / l rounded to bf16 and the split's log2-domain
            // lse; register order, two accumulator groups (16 bytes) per
            // lane, so each store instruction writes 1 KB contiguous.
            // Partials are stored non-temporally (read once, by the combine
            // launch)
            const int64_t blk = (((int64_t)split * a.B + b) * a.Hkv + kvh) * a.nrb + (r >> 5);
            const float inv = lt > 0.f ? 1.f / lt : 0.f;
            uint16_t *op = (uint16_t *)a.part_o + blk * (32 * D) + 8 * lane;
#pragma unroll
            for (int pg = 0; pg < 2 * MD; ++pg) {
                const int md = pg >> 1, g0 = 2 * (pg & 1);
                u32x4 val;
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    val[2 * h + 0] = pack_bf16x2(o[n][md][4 * (g0 + h) + 0] * inv, o[n][md][4 * (g0 + h) + 1] * inv);
                    val[2 * h + 1] = pack_bf16x2(o[n][md][4 * (g0 + h) + 2] * inv, o[n][md][4 * (g0 + h) + 3] * inv);
                }
                __builtin_nontemporal_store(val, (u32x4 *)(op + pg * 512));
            }
            if (hf == 0) __builtin_nontemporal_store(lt > 0.f ? m[n] + __builtin_amdgcn_logf(lt) : -INFINITY, a.part_ml + blk * 32 + l32);
        } else {
            // register order: each store instruction writes 1 KB contiguous
            const int64_t blk = (((int64_t)split * a.B + b) * a.Hkv + kvh) * a.nrb + (r >> 5);
            float *op = a.part_o + blk * (32 * D) + 4 * lane;
#pragma unroll
            for (int md = 0; md < MD; ++md)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    f32x4 val;
#pragma unroll
                    for (int e = 0; e < 4; ++e) val[e] = o[n][md][4 * g + e];
                    __builtin_nontemporal_store(val, (f32x4 *)(op + (md * 4 + g) * 256));
                }
            if (hf == 0) {
                __builtin_nontemporal_store(m[n], a.part_ml + 2 * (blk * 32 + l32) + 0);
                __builtin_nontemporal_store(lt, a.part_ml + 2 * (blk * 32 + l32) + 1);
            }
        }
    }

    // ---- fused append -----------------------------------------------------
    // Step items cover every query head of their KV group (packed rows),
    // so the items of a (stream, KV head) group split the new tokens evenly
    // among them; padding tokens (t >= nl) are not committed.
    // This kernel reads the new block from kc/vc, never from the slots being
    // written, so the append can trail the attention; it comes after the
    // epilogue's stores so that its loads overlap their drain.
    if (step && a.fuse_append && hh == 0)
        append_share<D, NT>(a, b, kvh, (int)(qi * a.nsplit + split), n_pool, nl, ptab, tid);
}

// bf16 output: split s holds o_s / l_s (bf16) and lse_s = m_s + log2(l_s);
//   M = max_s lse_s,  L = sum_s 2^(lse_s - M),  o = sum_s 2^(lse_s - M) o_s / L.
// A thread owns the 8 elements (two accumulator groups) one writer lane
// stored with one 16-byte store, for every split.
// VARLEN: blocks of different lengths; padding rows are skipped (their
// partials may not exist).  SMAX >= nsplit: the split loops are unrolled
// SMAX times (the launch takes the smallest of 8, 16, 32, which also keeps
// the register count, and with it the waves per SIMD that hide the loads'
// latency, down).
template <int D, bool VARLEN, int SMAX>
__global__ __launch_bounds__(256) void combine16_kernel(const AttnArgs a) {
    static_assert(SMAX <= MAX_SPLITS, "at most MAX_SPLITS partials");
    constexpr int MD = D / 32;
    constexpr int PER_BLK = 2 * MD * 64;      // 16-byte items per 32-row block
    const int64_t nblk = (int64_t)a.B * a.Hkv * a.nrb;
    const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (u >= nblk * PER_BLK) return;
    const int64_t blk = u / PER_BLK;
    const int item = (int)(u % PER_BLK);
    const int lane = item & 63;
    const int pg = item >> 6;                 // md * 2 + g0 / 2
    const int r = (int)(blk % a.nrb) * 32 + (lane & 31);   // packed row
    if (r >= a.nrows) return;
    const int kvh = (int)((blk / a.nrb) % a.Hkv);
    const int b = (int)(blk / ((int64_t)a.nrb * a.Hkv));
    const int t = r / a.G;
    if (VARLEN && t >= a.new_lens[b]) return;   // padding row: left unwritten
    const int hq = kvh * a.G + (r - t * a.G);
    const int S = a.nsplit;
    const float *pl = a.part_ml + blk * 32 + (lane & 31);
    const uint16_t *po = (const uint16_t *)a.part_o + blk * (32 * D) + pg * 512 + 8 * lane;
    const int64_t ls = nblk * 32;             // split stride of lse
    const int64_t ps = nblk * 32 * D;         // split stride of o
    // all loads first (one round trip), then the arithmetic
    float lse[SMAX];
    u32x4 ov[SMAX];
#pragma unroll
    for (int s = 0; s < SMAX; ++s) {
        if (s < S) {
            lse[s] = pl[s * ls];
            ov[s] = *(const u32x4 *)(po + s * ps);
        } else {
            lse[s] = -INFINITY;
            ov[s] = u32x4{0u, 0u, 0u, 0u};
        }
    }
    float M = -INFINITY;
#pragma unroll
    for (int s = 0; s < SMAX; ++s) M = fmaxf(M, lse[s]);
    const float Mu = (M == -INFINITY) ? 0.f : M;
    float L = 0.f;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < SMAX; ++s) {
        const float wgt = __builtin_amdgcn_exp2f(lse[s] - Mu);   // 0 for absent splits
        L += wgt;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            acc[2 * k + 0] += __uint_as_float(ov[s][k] << 16) * wgt;
            acc[2 * k + 1] += __uint_as_float(ov[s][k] & 0xFFFF0000u) * wgt;
        }
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    const int md = pg >> 1, g0 = 2 * (pg & 1), hf = lane >> 5;
    uint16_t *op = (uint16_t *)a.out + b * a.o_sb + (int64_t)t * a.o_st + hq * a.o_sh + 32 * md + 4 * hf;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        u32x2 val;
        val[0] = pack_bf16x2(acc[4 * h + 0] * inv, acc[4 * h + 1] * inv);
        val[1] = pack_bf16x2(acc[4 * h + 2] * inv, acc[4 * h + 3] * inv);
        *(u32x2 *)(op + 8 * (g0 + h)) = val;
    }
    if (a.lse && pg == 0 && lane < 32)
        a.lse[((int64_t)b * a.Hq + hq) * a.Lq + t] = (M + __builtin_amdgcn_logf(L)) * 0.69314718055994531f;
}

// Merge the KV-split partials of every query row: with per-split running
// max m_s (log2 domain), sum l_s and unnormalised o_s,
//   M = max_s m_s,  L = sum_s l_s 2^(m_s - M),  o = sum_s o_s 2^(m_s - M) / L.
// Splits are visited in a fixed order, so the result is deterministic.  A
// thread owns the 4 elements one accumulator lane holds for one (md, g), so
// its partial reads are the writer's contiguous 1 KB runs; the split loops
// are unrolled so their independent loads are in flight together.
template <int D, bool VARLEN>
__global__ __launch_bounds__(256) void combine_kernel(const AttnArgs a) {
    constexpr int MD = D / 32;
    constexpr int PER_BLK = MD * 4 * 64;      // float4 items per 32-row block
    const int64_t nblk = (int64_t)a.B * a.Hkv * a.nrb;
    const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (u >= nblk * PER_BLK) return;
    const int64_t blk = u / PER_BLK;
    const int item = (int)(u % PER_BLK);
    const int lane = item & 63;
    const int mg = item >> 6;                 // md * 4 + g
    const int r = (int)(blk % a.nrb) * 32 + (lane & 31);   // packed row
    if (r >= a.nrows) return;
    const int kvh = (int)((blk / a.nrb) % a.Hkv);
    const int b = (int)(blk / ((int64_t)a.nrb * a.Hkv));
    const int t = r / a.G;
    if (VARLEN && t >= a.new_lens[b]) return;   // padding row: left unwritten
    const int hq = kvh * a.G + (r - t * a.G);
    const int d0 = 32 * (mg >> 2) + 8 * (mg & 3) + 4 * (lane >> 5);
    const int S = a.nsplit;
    const float2 *ml = (const float2 *)a.part_ml + blk * 32 + (lane & 31);
    const float *po = a.part_o + blk * (32 * D) + (int64_t)mg * 256 + 4 * lane;
    const int64_t mls = nblk * 32;            // split stride of (m, l)
    const int64_t ps = nblk * 32 * D;         // split stride of o
    float M = -INFINITY;
#pragma unroll 8
    for (int s = 0; s < S; ++s) M = fmaxf(M, ml[s * mls].x);
    const float Mu = (M == -INFINITY) ? 0.f : M;
    float L = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int s = 0; s < S; ++s) {
        const float2 m_l = ml[s * mls];
        const f32x4 ov = *(const f32x4 *)(po + s * ps);
        const float wgt = __builtin_amdgcn_exp2f(m_l.x - Mu);
        L += m_l.y * wgt;
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] += ov[e] * wgt;
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    if (a.out_f32) {
        float *op = (float *)a.out + b * a.o_sb + (int64_t)t * a.o_st + hq * a.o_sh + d0;
        f32x4 val;
#pragma unroll
        for (int e = 0; e < 4; ++e) val[e] = acc[e] * inv;
        *(f32x4 *)op = val;
    } else {
        uint16_t *op = (uint16_t *)a.out + b * a.o_sb + (int64_t)t * a.o_st + hq * a.o_sh + d0;
        u32x2 val;
        val[0] = pack_bf16x2(acc[0] * inv, acc[1] * inv);
        val[1] = pack_bf16x2(acc[2] * inv, acc[3] * inv);
        *(u32x2 *)op = val;
    }
    if (a.lse && mg == 0 && lane < 32)
        a.lse[((int64_t)b * a.Hq + hq) * a.Lq + t] = (M + __builtin_amdgcn_logf(L)) * 0.69314718055994531f;
}

// Copy new tokens' K/V rows into their cache slots: one 16-byte chunk per
// thread; consecutive threads walk one token row, so reads and writes are
// contiguous 256-byte runs (head_dim 128).
__global__ __launch_bounds__(256) void append_kernel(const AppendArgs a) {
    const int CH = a.D / 8;
    const int b = blockIdx.y;
    const int64_t total = (int64_t)(a.new_lens ? a.new_lens[b] : a.Ln) * a.Hkv * CH;
    for (int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x; u < total; u += (int64_t)gridDim.x * 256) {
        const int c = (int)(u % CH);
        const int h = (int)((u / CH) % a.Hkv);
        const int t = (int)(u / ((int64_t)CH * a.Hkv));
        const int pos = a.cache_lens[b] + t;
        const int page = a.page_table[(int64_t)b * a.max_pages + (pos >> 6)];
        const int64_t dst = (((int64_t)page * a.Hkv + h) * KT + (pos & 63)) * a.D + 8 * c;
        *(u32x4 *)(a.kpool + dst) = *(const u32x4 *)(a.kn + b * a.kn_sb + (int64_t)t * a.kn_st + h * a.kn_sh + 8 * c);
        *(u32x4 *)(a.vpool + dst) = *(const u32x4 *)(a.vn + b * a.vn_sb + (int64_t)t * a.vn_st + h * a.vn_sh + 8 * c);
    }
}

template <int D, int NW, int NB>
int launch_attn_t(const AttnArgs &a, hipStream_t st) {
    const int grid = a.per_xcd * NUM_XCD;
    hipLaunchKernelGGL((attn_kernel<D, NW, NB>), dim3(grid), dim3(NW * 64), 0, st, a);
    return (int)hipGetLastError();
}

}  // namespace

int launch_attention(const AttnArgs &a, int head_dim, TileShape shape, void *stream) {
    hipStream_t st = (hipStream_t)stream;
    if (shape.nw != 8 || shape.nb != 1) return (int)hipErrorInvalidValue;
    if (head_dim == 128) return launch_attn_t<128, 8, 1>(a, st);
    if (head_dim == 64) return launch_attn_t<64, 8, 1>(a, st);
    return (int)hipErrorInvalidValue;
}

typedef void (*CombineKern)(const AttnArgs);

template <int D, bool VL>
CombineKern combine16_for(int nsplit) {
    return nsplit <= 8 ? combine16_kernel<D, VL, 8>
         : nsplit <= 16 ? combine16_kernel<D, VL, 16> : combine16_kernel<D, VL, MAX_SPLITS>;
}

int launch_combine(const AttnArgs &a, int head_dim, void *stream) {
    hipStream_t st = (hipStream_t)stream;
    typedef CombineKern Kern;
    const bool vl = a.has_new_lens != 0;
    if (!a.out_f32) {
        const int64_t items = (int64_t)a.B * a.Hkv * a.nrb * (head_dim / 32) * 2 * 64;
        const int64_t grid = (items + 255) / 256;
        Kern k = head_dim == 128 ? (vl ? combine16_for<128, true>(a.nsplit) : combine16_for<128, false>(a.nsplit))
                                 : (vl ? combine16_for<64, true>(a.nsplit) : combine16_for<64, false>(a.nsplit));
        hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(256), 0, st, a);
        return (int)hipGetLastError();
    }
    const int64_t items = (int64_t)a.B * a.Hkv * a.nrb * (head_dim / 32) * 4 * 64;
    const int64_t grid = (items + 255) / 256;
    Kern k = head_dim == 128 ? (vl ? combine_kernel<128, true> : combine_kernel<128, false>)
                             : (vl ? combine_kernel<64, true> : combine_kernel<64, false>);
    hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(256), 0, st, a);
    return (int)hipGetLastError();
}

int launch_append(const AppendArgs &a, void *stream) {
    hipStream_t st = (hipStream_t)stream;
    const int64_t total = (int64_t)a.Ln * a.Hkv * (a.D / 8);
    int64_t gx = (total + 255) / 256;
    if (gx > 4096) gx = 4096;
    if (gx < 1) gx = 1;
    hipLaunchKernelGGL(append_kernel, dim3((unsigned)gx, (unsigned)a.B), dim3(256), 0, st, a);
    return (int)hipGetLastError();
}


}  // namespace ws
