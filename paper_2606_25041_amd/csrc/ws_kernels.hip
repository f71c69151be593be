// gfx950 (MI355X) kernels for block-causal streaming attention.
//
// Block-causal rule (Wan-Streamer v0.1, Abstract; Sec. 1 with Fig. 1): a
// token sees its whole own block and every earlier block.  The step kernel
// runs the performer's current unit against its full-history cache
// (Sec. 2.4); the prefill kernel covers whole sequences (Sec. 2.4, system
// prefill); the append kernel commits a KV slice to the paged cache
// (Sec. 2.4).
//
// Attention kernel design (one work-group = one (stream, query head,
// query tile, KV split) work item; waves own 32*NB query rows each):
//  * S^T = K Q^T on v_mfma_f32_32x32x16_bf16: K (A operand) from LDS, Q (B
//    operand) resident in registers.  In the 32x32 accumulator layout a lane
//    owns one query column and 16 keys, so row max/sum are in-lane plus one
//    v_permlane32_swap per 64-key tile.
//  * Online softmax in the log2 domain (scale*log2(e) folded into one FMA),
//    fp32 running max/sum per lane.
//  * O^T += V^T P^T on the same MFMA: P stays in registers (the accumulator
//    layout of S^T is exactly the B-operand layout once the 16 keys of each
//    MFMA step are permuted consistently on both operands); V is read with
//    ds_read_b64_tr_b16 from a row-major LDS tile, so no transpose pass.
//    Each lane owns one query column of O^T, so the softmax rescale is a
//    per-lane scalar multiply.
//  * K/V tiles of 64 keys (= one cache page) are staged global -> VGPR ->
//    LDS with 128-bit loads, double-buffered in LDS (one barrier per tile),
//    the next tile's loads in flight during the current tile's MFMAs.
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

namespace ws {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int KT = 64;        // keys per tile (= page size)
constexpr int NUM_XCD = 8;    // MI355X: 8 XCDs, work-groups dispatched round-robin
constexpr float RESCALE_LOG2 = 8.f;  // lazy-rescale threshold (log2 units)
constexpr int PAGE_LDS = 2560;       // page ids of a split staged in LDS (more: read from memory)

typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// max / sum of a value over lanes l and l^32 (same query column, other keys)
__device__ __forceinline__ float halves_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// End (exclusive) of the block that holds token i: the first offset > i.
__device__ __forceinline__ int block_end(const int32_t *off, int nb, int i) {
    int lo = 1, hi = nb;  // answer index in [1, nb]
    while (lo < hi) {
        int mid = (lo + hi) >> 1;
        if (off[mid] > i) hi = mid; else lo = mid + 1;
    }
    return off[lo];
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    __bf16 a = (__bf16)lo, b = (__bf16)hi;
    return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

template <int D, int NB, int NW>
__global__ __launch_bounds__(NW * 64) void attn_kernel(const AttnArgs a) {
    constexpr int NT = NW * 64;
    constexpr int QT = NW * 32 * NB;
    constexpr int CH = D / 8;             // 16-byte chunks per key row
    constexpr int KP = D * 2 + 16;        // K row pitch in LDS (bytes): conflict-free b128 reads
    constexpr int VP = D * 2 + 32;        // V row pitch in LDS (bytes): conflict-free transpose reads
    constexpr int KBYTES = KT * KP;
    constexpr int VBYTES = KT * VP;
    constexpr int LOADS = KT * CH / NT;   // 16-byte chunks per thread per tile, each of K and V
    constexpr int KK = D / 16;            // MFMA k-steps over head_dim for S
    constexpr int MD = D / 32;            // 32-row blocks of head_dim for O^T
    static_assert((KT * CH) % NT == 0, "tile chunks must divide among threads");
    __shared__ __attribute__((aligned(16))) char smem[2 * (KBYTES + VBYTES)];
    __shared__ int page_lds[PAGE_LDS];

    // ---- work item ------------------------------------------------------
    const int bid = blockIdx.x;
    const int w = (bid % NUM_XCD) * a.per_xcd + bid / NUM_XCD;
    if (w >= a.n_work) return;
    const int per_group = a.G * a.nqt * a.nsplit;
    const int group = w / per_group;
    const int idx = w - group * per_group;
    const int qi = idx / (a.G * a.nsplit);
    const int rem = idx - qi * (a.G * a.nsplit);
    const int split = rem / a.G;
    const int hh = rem - split * a.G;
    const int b = group / a.Hkv;
    const int kvh = group - b * a.Hkv;
    const int hq = kvh * a.G + hh;
    const bool step = a.mode == MODE_STEP;
    const int qt = step ? qi : (a.nqt - 1 - qi);  // prefill: heaviest tiles first
    const int q0 = qt * QT;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int hf = lane >> 5;     // which half of the wave
    const int l32 = lane & 31;

    // ---- key range ------------------------------------------------------
    const int32_t *offs = step ? nullptr : a.offsets + (int64_t)b * (a.nb + 1);
    int n_pool, k_hi, kfull;
    if (step) {
        n_pool = (a.lens_in_args && b < LENS_IN_ARGS) ? a.lens_arg[b] : a.cache_lens[b];
        k_hi = n_pool + a.Lq;
        kfull = k_hi;
    } else {
        n_pool = a.paged ? a.Lq : 0;
        const int q_last = min(q0 + QT, a.Lq) - 1;
        k_hi = block_end(offs, a.nb, q_last);
        kfull = block_end(offs, a.nb, q0);
    }
    const int ntile = (k_hi + KT - 1) / KT;
    const int t_begin = (int)((int64_t)split * ntile / a.nsplit);
    const int t_end = (int)((int64_t)(split + 1) * ntile / a.nsplit);

    // ---- this lane's query rows -----------------------------------------
    int rows[NB], kend[NB];
    bf16x8 qf[NB][KK];
#pragma unroll
    for (int n = 0; n < NB; ++n) {
        rows[n] = q0 + wave * 32 * NB + n * 32 + l32;
        const int rc = min(rows[n], a.Lq - 1);
        kend[n] = step ? k_hi : block_end(offs, a.nb, rc);
        const uint16_t *qp = a.q + b * a.q_sb + (int64_t)rc * a.q_st + hq * a.q_sh + 8 * hf;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) qf[n][kk] = *(const bf16x8 *)(qp + 16 * kk);
    }

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

    // ---- tile staging ---------------------------------------------------
    // Physical pages of the cache tiles: the first three are loaded at entry
    // as independent loads (so the first K/V loads wait on one page-table
    // read only); the rest of the split's page ids are staged in LDS before
    // the first barrier, so no page-table read sits in front of a later tile.
    const int32_t *ptab = a.page_table + (int64_t)b * a.max_pages;
    const int tp_end = min(t_end, (n_pool + KT - 1) / KT);   // tiles with cache rows
    auto page_glb = [&](int t) -> int { return t < tp_end ? ptab[t] : 0; };
    const int pg0 = page_glb(t_begin), pg1 = page_glb(t_begin + 1), pg2 = page_glb(t_begin + 2);
    const int n_lds_pages = min(max(tp_end - t_begin, 0), PAGE_LDS);
    int pre[PAGE_LDS / NT];
#pragma unroll
    for (int k = 0; k < PAGE_LDS / NT; ++k) {
        const int i = tid + k * NT;
        pre[k] = i < n_lds_pages ? ptab[t_begin + i] : 0;
    }
    auto page_of = [&](int t) -> int {
        const int i = t - t_begin;
        return i < PAGE_LDS ? page_lds[i] : page_glb(t);
    };

    // Fused append, first round: this thread's chunk of the new block is
    // loaded now and written after the prologue, off the critical path.  The
    // G query heads of a group share one KV head, so only the items of its
    // first head write; they split the new tokens evenly among them.
    const bool appends = step && a.fuse_append && hh == 0;
    int app_s0 = 0, app_n = 0;
    if (appends) {
        const int napp = a.nqt * a.nsplit;
        const int ai = qi * a.nsplit + split;
        app_s0 = (int)((int64_t)ai * a.Lq / napp);
        app_n = ((int)((int64_t)(ai + 1) * a.Lq / napp) - app_s0) * CH;
    }
    auto app_src = [&](int u, int64_t &src_k, int64_t &src_v, int &pos, int &c) {
        const int t = app_s0 + u / CH;
        c = u % CH;
        pos = n_pool + t;
        src_k = b * a.kc_sb + (int64_t)t * a.kc_st + kvh * a.kc_sh + 8 * c;
        src_v = b * a.vc_sb + (int64_t)t * a.vc_st + kvh * a.vc_sh + 8 * c;
    };
    auto app_dst = [&](int page, int pos, int c) -> int64_t {
        return (((int64_t)page * a.Hkv + kvh) * KT + (pos & 63)) * D + 8 * c;
    };
    u32x4 app_k = {0, 0, 0, 0}, app_v = {0, 0, 0, 0};
    int app_page = 0, app_pos = 0, app_c = 0;
    const bool app_first = tid < app_n;
    if (app_first) {
        int64_t sk, sv;
        app_src(tid, sk, sv, app_pos, app_c);
        app_page = ptab[app_pos >> 6];
        app_k = *(const u32x4 *)(a.kc + sk);
        app_v = *(const u32x4 *)(a.vc + sv);
    }
    // Per-thread parts of the K/V addresses, fixed for the whole loop: this
    // thread stages chunk c of rows row0 + i * (NT / CH) of every tile.
    constexpr int RSTEP = NT / CH;
    const int row0 = tid / CH;
    const int cchunk = tid % CH;
    const int64_t page_elems = (int64_t)a.Hkv * KT * D;
    const uint16_t *kpool_t = a.kpool + ((int64_t)kvh * KT + row0) * D + 8 * cchunk;
    const uint16_t *vpool_t = a.vpool + ((int64_t)kvh * KT + row0) * D + 8 * cchunk;
    const uint16_t *kc_t = a.kc + b * a.kc_sb + kvh * a.kc_sh + 8 * cchunk;
    const uint16_t *vc_t = a.vc + b * a.vc_sb + kvh * a.vc_sh + 8 * cchunk;
    // Two staging sets: the loads of tiles t+1 and t+2 are in flight while
    // tile t is computed from LDS.
    u32x4 kA[LOADS], vA[LOADS], kB[LOADS], vB[LOADS];
    auto load_tile = [&](int kt, int page, u32x4 (&kreg)[LOADS], u32x4 (&vreg)[LOADS]) {
        if (kt + KT <= n_pool) {
            // whole tile in one cache page
            const int64_t po = (int64_t)page * page_elems;
#pragma unroll
            for (int i = 0; i < LOADS; ++i) {
                kreg[i] = *(const u32x4 *)(kpool_t + po + i * RSTEP * D);
                vreg[i] = *(const u32x4 *)(vpool_t + po + i * RSTEP * D);
            }
        } else if (kt >= n_pool && kt + KT <= k_hi) {
            // whole tile in the contiguous keys
            const int64_t j0 = kt - n_pool + row0;
#pragma unroll
            for (int i = 0; i < LOADS; ++i) {
                kreg[i] = *(const u32x4 *)(kc_t + (j0 + i * RSTEP) * a.kc_st);
                vreg[i] = *(const u32x4 *)(vc_t + (j0 + i * RSTEP) * a.vc_st);
            }
        } else {
            // the tile straddles the cache end or runs past the last key:
            // rows past the end repeat a valid row (their scores are masked)
#pragma unroll
            for (int i = 0; i < LOADS; ++i) {
                const int j = min(kt + row0 + i * RSTEP, k_hi - 1);
                if (j < n_pool) {
                    const int64_t po = (int64_t)page * page_elems + (int64_t)((j & 63) - row0) * D;
                    kreg[i] = *(const u32x4 *)(kpool_t + po);
                    vreg[i] = *(const u32x4 *)(vpool_t + po);
                } else {
                    kreg[i] = *(const u32x4 *)(kc_t + (int64_t)(j - n_pool) * a.kc_st);
                    vreg[i] = *(const u32x4 *)(vc_t + (int64_t)(j - n_pool) * a.vc_st);
                }
            }
        }
    };
    auto store_tile = [&](int buf, const u32x4 (&kreg)[LOADS], const u32x4 (&vreg)[LOADS]) {
        char *ks = smem + buf * (KBYTES + VBYTES) + row0 * KP + 16 * cchunk;
        char *vs = smem + buf * (KBYTES + VBYTES) + KBYTES + row0 * VP + 16 * cchunk;
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            *(u32x4 *)(ks + i * RSTEP * KP) = kreg[i];
            *(u32x4 *)(vs + i * RSTEP * VP) = vreg[i];
        }
    };

    const float c2 = a.scale_log2;

    auto compute_tile = [&](int buf, int kt) {
        const char *ks = smem + buf * (KBYTES + VBYTES);
        const char *vs = ks + KBYTES;
        // S^T[key][query] = K Q^T for 64 keys x (32*NB) queries of this wave
        f32x16 s[2][NB];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int n = 0; n < NB; ++n)
#pragma unroll
                for (int v = 0; v < 16; ++v) s[mb][n][v] = 0.f;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) {
                const bf16x8 ka = *(const bf16x8 *)(ks + (mb * 32 + l32) * KP + (16 * kk + 8 * hf) * 2);
#pragma unroll
                for (int n = 0; n < NB; ++n)
                    s[mb][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[n][kk], s[mb][n], 0, 0, 0);
            }
        }

        // element masks only where the tile is not visible to every row
        if (kt + KT > kfull) {
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int key = kt + mb * 32 + (v >> 2) * 8 + 4 * hf + (v & 3);
#pragma unroll
                    for (int n = 0; n < NB; ++n)
                        if (key >= kend[n]) s[mb][n][v] = -INFINITY;
                }
        }

        // online softmax (log2 domain)
        bf16x8 pf[NB][4];
#pragma unroll
        for (int n = 0; n < NB; ++n) {
            float mx = -INFINITY;
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[mb][n][v]);
            mx = halves_max(mx) * c2;
            // Lazy rescale: the running max m only moves when the tile max
            // exceeds it by more than 2^RESCALE_LOG2, so most tiles skip the
            // rescale of O and l (a wave-uniform branch).  Weights stay
            // <= 2^RESCALE_LOG2; O and l share the same m, so the final
            // quotient is unchanged.
            const bool grow = mx > m[n] + RESCALE_LOG2;
            if (__builtin_amdgcn_ballot_w64(grow)) {
                const float m_new = grow ? mx : m[n];
                const float alpha = fast_exp2(m[n] - m_new);  // 1 where m is kept; 0 from -inf
                m[n] = m_new;
                l[n] *= alpha;
#pragma unroll
                for (int md = 0; md < MD; ++md)
#pragma unroll
                    for (int v = 0; v < 16; ++v) o[n][md][v] *= alpha;
            }
            const float m_use = (m[n] == -INFINITY) ? 0.f : m[n];
            float rs = 0.f;
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const float p = fast_exp2(__builtin_fmaf(s[mb][n][v], c2, -m_use));
                    s[mb][n][v] = p;
                    rs += p;
                }
            l[n] += rs;
#pragma unroll
            for (int ks4 = 0; ks4 < 4; ++ks4)
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    pf[n][ks4][e] = (__bf16)s[ks4 >> 1][n][8 * (ks4 & 1) + e];
        }

        // O^T[d][query] += V^T P^T; V^T fragments by LDS transpose reads
        const int j16 = lane & 15;
        const int dsub = 16 * ((lane >> 4) & 1) + 4 * (j16 & 3);
#pragma unroll
        for (int ks4 = 0; ks4 < 4; ++ks4) {
            const int k0 = 16 * ks4 + 4 * hf + (j16 >> 2);
#pragma unroll
            for (int md = 0; md < MD; ++md) {
                const int dcol = 32 * md + dsub;
                const i16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_i16x4 *)(vs + k0 * VP + dcol * 2));
                const i16x4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_i16x4 *)(vs + (k0 + 8) * VP + dcol * 2));
                // whole-vector reinterpretation: element-wise bf16 casts of
                // the transpose-read result were lowered to a splat
                const bf16x8 vfrag = __builtin_bit_cast(
                    bf16x8, __builtin_shufflevector(va, vb, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
                for (int n = 0; n < NB; ++n)
                    o[n][md] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfrag, pf[n][ks4], o[n][md], 0, 0, 0);
            }
        }

    };

    // Pipeline: tile t is computed from LDS buffer (t - t_begin) & 1 while
    // the loads of tiles t+1 and t+2 are in flight in the two register sets;
    // after the compute, tile t+1 is stored to the other buffer and the loads
    // of tile t+3 are issued.  One barrier per tile.  Unrolled by two so the
    // register set of every step is fixed at compile time.
    // Prologue: only the first tile is requested before the first compute,
    // so it is not queued behind the next tiles of every other work-group;
    // tiles 1 and 2 stream in while tile 0 is computed.
    if (t_begin < t_end) {
        load_tile(t_begin * KT, pg0, kA, vA);
        store_tile(0, kA, vA);
        if (t_begin + 1 < t_end) load_tile((t_begin + 1) * KT, pg1, kB, vB);
        if (t_begin + 2 < t_end) load_tile((t_begin + 2) * KT, pg2, kA, vA);
    }
#pragma unroll
    for (int k = 0; k < PAGE_LDS / NT; ++k)
        if (tid + k * NT < n_lds_pages) page_lds[tid + k * NT] = pre[k];
    if (app_first) {
        const int64_t dst = app_dst(app_page, app_pos, app_c);
        *(u32x4 *)(a.kpool + dst) = app_k;
        *(u32x4 *)(a.vpool + dst) = app_v;
    }
    __syncthreads();
    for (int t = t_begin; t < t_end; t += 2) {
        compute_tile(0, t * KT);
        if (t + 1 < t_end) store_tile(1, kB, vB);
        if (t + 3 < t_end) load_tile((t + 3) * KT, page_of(t + 3), kB, vB);
        __syncthreads();
        if (t + 1 >= t_end) break;
        compute_tile(1, (t + 1) * KT);
        if (t + 2 < t_end) store_tile(0, kA, vA);
        if (t + 4 < t_end) load_tile((t + 4) * KT, page_of(t + 4), kA, vA);
        __syncthreads();
    }

    // fused append, remaining rounds (more chunks than threads)
    for (int u = tid + NT; u < app_n; u += NT) {
        int64_t sk, sv;
        int pos, c;
        app_src(u, sk, sv, pos, c);
        const int64_t dst = app_dst(ptab[pos >> 6], pos, c);
        *(u32x4 *)(a.kpool + dst) = *(const u32x4 *)(a.kc + sk);
        *(u32x4 *)(a.vpool + dst) = *(const u32x4 *)(a.vc + sv);
    }

    // ---- epilogue -------------------------------------------------------
#pragma unroll
    for (int n = 0; n < NB; ++n) {
        const float lt = halves_sum(l[n]);
        const int r = rows[n];
        if (r >= a.Lq) continue;
        if (a.nsplit == 1) {
            const float inv = lt > 0.f ? 1.f / lt : 0.f;
            if (a.out_f32) {
                float *op = (float *)a.out + b * a.o_sb + (int64_t)r * a.o_st + hq * a.o_sh;
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
                uint16_t *op = (uint16_t *)a.out + b * a.o_sb + (int64_t)r * a.o_st + hq * a.o_sh;
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
                a.lse[((int64_t)b * a.Hq + hq) * a.Lq + r] = (m[n] + __builtin_amdgcn_logf(lt)) * 0.69314718055994531f;
        } else {
            // register order: each store instruction writes 1 KB contiguous
            const int64_t blk = (((int64_t)split * a.B + b) * a.Hq + hq) * a.nrb + (r >> 5);
            float *op = a.part_o + blk * (32 * D) + 4 * lane;
#pragma unroll
            for (int md = 0; md < MD; ++md)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    f32x4 val;
#pragma unroll
                    for (int e = 0; e < 4; ++e) val[e] = o[n][md][4 * g + e];
                    *(f32x4 *)(op + (md * 4 + g) * 256) = val;
                }
            if (hf == 0) {
                a.part_ml[2 * (blk * 32 + l32) + 0] = m[n];
                a.part_ml[2 * (blk * 32 + l32) + 1] = lt;
            }
        }
    }
}

// Merge the KV-split partials of every query row: with per-split running
// max m_s (log2 domain), sum l_s and unnormalised o_s,
//   M = max_s m_s,  L = sum_s l_s 2^(m_s - M),  o = sum_s o_s 2^(m_s - M) / L.
// Splits are visited in a fixed order, so the result is deterministic.  A
// thread owns the 4 elements one accumulator lane holds for one (md, g), so
// its partial reads are the writer's contiguous 1 KB runs; the split loops
// are unrolled so their independent loads are in flight together.
template <int D>
__global__ __launch_bounds__(256) void combine_kernel(const AttnArgs a) {
    constexpr int MD = D / 32;
    constexpr int PER_BLK = MD * 4 * 64;      // float4 items per 32-row block
    const int64_t nblk = (int64_t)a.B * a.Hq * a.nrb;
    const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (u >= nblk * PER_BLK) return;
    const int64_t blk = u / PER_BLK;
    const int item = (int)(u % PER_BLK);
    const int lane = item & 63;
    const int mg = item >> 6;                 // md * 4 + g
    const int r = (int)(blk % a.nrb) * 32 + (lane & 31);
    if (r >= a.Lq) return;
    const int hq = (int)((blk / a.nrb) % a.Hq);
    const int b = (int)(blk / ((int64_t)a.nrb * a.Hq));
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
        float *op = (float *)a.out + b * a.o_sb + (int64_t)r * a.o_st + hq * a.o_sh + d0;
        f32x4 val;
#pragma unroll
        for (int e = 0; e < 4; ++e) val[e] = acc[e] * inv;
        *(f32x4 *)op = val;
    } else {
        uint16_t *op = (uint16_t *)a.out + b * a.o_sb + (int64_t)r * a.o_st + hq * a.o_sh + d0;
        u32x2 val;
        val[0] = pack_bf16x2(acc[0] * inv, acc[1] * inv);
        val[1] = pack_bf16x2(acc[2] * inv, acc[3] * inv);
        *(u32x2 *)op = val;
    }
    if (a.lse && mg == 0 && lane < 32)
        a.lse[((int64_t)b * a.Hq + hq) * a.Lq + r] = (M + __builtin_amdgcn_logf(L)) * 0.69314718055994531f;
}

// Copy new tokens' K/V rows into their cache slots: one 16-byte chunk per
// thread; consecutive threads walk one token row, so reads and writes are
// contiguous 256-byte runs (head_dim 128).
__global__ __launch_bounds__(256) void append_kernel(const AppendArgs a) {
    const int CH = a.D / 8;
    const int64_t total = (int64_t)a.Ln * a.Hkv * CH;
    const int b = blockIdx.y;
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

template <int D, int NB, int NW>
int launch_attn_t(const AttnArgs &a, hipStream_t st) {
    const int grid = a.per_xcd * NUM_XCD;
    hipLaunchKernelGGL((attn_kernel<D, NB, NW>), dim3(grid), dim3(NW * 64), 0, st, a);
    return (int)hipGetLastError();
}

}  // namespace

int launch_attention(const AttnArgs &a, int head_dim, TileShape shape, void *stream) {
    hipStream_t st = (hipStream_t)stream;
    if (shape.nb != 1) return (int)hipErrorInvalidValue;
    if (head_dim == 128) {
        if (shape.nw == 4) return launch_attn_t<128, 1, 4>(a, st);
        if (shape.nw == 8) return launch_attn_t<128, 1, 8>(a, st);
    } else if (head_dim == 64) {
        if (shape.nw == 4) return launch_attn_t<64, 1, 4>(a, st);
        if (shape.nw == 8) return launch_attn_t<64, 1, 8>(a, st);
    }
    return (int)hipErrorInvalidValue;
}

int launch_combine(const AttnArgs &a, int head_dim, void *stream) {
    hipStream_t st = (hipStream_t)stream;
    const int64_t items = (int64_t)a.B * a.Hq * a.nrb * (head_dim / 32) * 4 * 64;
    const int64_t grid = (items + 255) / 256;
    if (head_dim == 128)
        hipLaunchKernelGGL(combine_kernel<128>, dim3((unsigned)grid), dim3(256), 0, st, a);
    else
        hipLaunchKernelGGL(combine_kernel<64>, dim3((unsigned)grid), dim3(256), 0, st, a);
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
