// gfx950 (MI355X) kernels for the gradients of whole-sequence block-causal
// attention (training uses the same causal format as generation,
// Wan-Streamer v0.1, Sec. 2.3): a per-row prep pass, a query-major dQ kernel
// and a key-major dK/dV kernel, all deterministic.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ws_kernels.h"
#include "ws_device_util.h"

namespace ws {
namespace {

constexpr int KB_DKDV = 16;   // key tiles of one group taken together on an XCD (dK/dV)

// ---------------------------------------------------------------------------
// Gradients of the whole-sequence path (training shares the causal format,
// Sec. 2.3).  With the forward's lse, P_ij = exp(s_ij - lse_i) needs no
// running max:
//   D_i = <dO_i, O_i>,  dS_ij = P_ij (<dO_i, v_j> - D_i),
//   dQ_i = scale sum_j dS_ij k_j,  dK_j = scale sum_i dS_ij q_i,
//   dV_j = sum_i P_ij dO_i.
// Two kernels after a per-row prep pass: a query-major one for dQ (like the
// forward, with dS^T in place of P^T) and a key-major one for dK and dV
// (S = Q K^T with the keys as columns, so P and dS are B operands of
// dV^T += dO^T P and dK^T += Q^T dS).  Each sums in a fixed order: the
// gradients are deterministic, and dK/dV sum the G query heads of their KV
// head inside one work-group.

// byte offset of 16-byte chunk c of row r in an LDS tile of [rows][D] bf16
// (the forward's swizzle)
template <int D>
__device__ __forceinline__ uint32_t tile_off(int r, int c) {
    return (uint32_t)(r * 2 * D + 16 * (c ^ swz<D>(r)));
}

// A fragment of (tile rows 16 ks .. 16 ks + 15)^T for head-dim block md, by
// two transpose reads; tb[] are the lane's bases (as the forward's V^T reads)
template <int D>
__device__ __forceinline__ bf16x8 tr_frag(const char *tile, const uint32_t (&tb)[2], int ks, int md) {
    const i16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4 *)(tile + ks * 16 * 2 * D + (tb[0] ^ (64 * md))));
    const i16x4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4 *)(tile + ks * 16 * 2 * D + (tb[1] ^ (64 * md))));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(va, vb, 0, 1, 2, 3, 4, 5, 6, 7));
}

template <int D>
__device__ __forceinline__ void tr_bases(int lane, uint32_t (&tb)[2]) {
    const int j16 = lane & 15, hf = lane >> 5;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const int vr = 4 * hf + (j16 >> 2) + 8 * e;
        const int vc = 2 * ((lane >> 4) & 1) + ((j16 & 3) >> 1);
        tb[e] = (uint32_t)(vr * 2 * D + 16 * (vc ^ swz<D>(vr)) + 8 * (j16 & 1));
    }
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Per row: (lse * log2(e), <dO, O>) and, per token, the end of the keys it
// sees.  LPR lanes per row, 16 bytes each.
template <int D>
__global__ __launch_bounds__(256) void bwd_prep_kernel(const BwdArgs a) {
    constexpr int LPR = D / 8;
    constexpr int RPB = 256 / LPR;
    const int64_t nrows = (int64_t)a.B * a.L * a.Hq;
    const int64_t r = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR;
    const int c = threadIdx.x % LPR;
    float part = 0.f;
    int h = 0, i = 0, b = 0;
    if (r < nrows) {
        h = (int)(r % a.Hq);
        i = (int)((r / a.Hq) % a.L);
        b = (int)(r / ((int64_t)a.Hq * a.L));
        const u32x4 ov = *(const u32x4 *)(a.o + b * a.o_sb + (int64_t)i * a.o_st + h * a.o_sh + 8 * c);
        const u32x4 dv = *(const u32x4 *)(a.dout + b * a.do_sb + (int64_t)i * a.do_st + h * a.do_sh + 8 * c);
#pragma unroll
        for (int k = 0; k < 4; ++k) part += bf16_lo(ov[k]) * bf16_lo(dv[k]) + bf16_hi(ov[k]) * bf16_hi(dv[k]);
    }
#pragma unroll
    for (int m = LPR / 2; m >= 1; m >>= 1) part += __shfl_xor(part, m, LPR);
    if (r < nrows && c == 0) {
        const int64_t idx = ((int64_t)b * a.Hq + h) * a.L + i;
        a.dl[2 * idx] = a.lse[idx] * 1.4426950408889634f;
        a.dl[2 * idx + 1] = part;
        if (h == 0) {
            const int32_t *offs = a.offsets + (int64_t)b * (a.nb + 1);
            const int32_t *text = a.text_starts ? a.text_starts + (int64_t)b * a.nb : nullptr;
            a.kend[(int64_t)b * a.L + i] = row_key_end<false>(offs, text, a.nb, i);
        }
    }
}

// Loads rows [r0, r0 + nrows) of a [rows][D] bf16 tile (row r of the tile
// = global row min(r0 + r, rmax), at least 0) straight into LDS at `lds` in the
// swizzled layout, spread over NWV waves: wave-wide load i of wave w fills
// tile bytes [(i * NWV + w) * 1024, +1024), lane l the 16 bytes at +16 l,
// so it fetches the chunk that belongs there.  The caller waits for them
// (s_waitcnt vmcnt) before the barrier that publishes the tile.
template <int D, int NWV, int ROWS>
__device__ __forceinline__ void dma_rows(const char *g, int64_t st_bytes, int r0, int rmax, uint32_t lds,
                                         int wave, int lane) {
    constexpr int ROWB = 2 * D, RPW = 1024 / ROWB, LPR = ROWB / 16;
    constexpr int NI = ROWS * ROWB / (NWV * 1024);
    static_assert(NI >= 1 && ROWS * ROWB % (NWV * 1024) == 0, "the tile splits into wave-wide loads");
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        const int r = (i * NWV + wave) * RPW + lane / LPR;
        const int ch = (lane % LPR) ^ swz<D>(r);
        const int gr = max(min(r0 + r, rmax), 0);
        dma16(g + (int64_t)gr * st_bytes + 16 * ch, lds + (i * NWV + wave) * 1024);
    }
}

// dQ: one work-group = (stream, query head, 128 query rows), 4 waves x 32
// rows; K/V tiles of 64 keys go straight to LDS (two stages); tiles past
// the last row's key end are never loaded.  Registers are held to two waves
// per SIMD, so two work-groups share a CU and one's softmax arithmetic runs
// beside the other's MFMAs.
template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void bwd_dq_kernel(const BwdArgs a) {
    constexpr int ROWB = 2 * D, KK = D / 16, MD = D / 32;
    constexpr int TILEB = 64 * ROWB;
    __shared__ __attribute__((aligned(1024))) char smem[2 * 2 * TILEB];   // [stage][K, V]
    const int nqt = (a.L + 127) / 128;
    const int wid = blockIdx.x;
    // query tiles heaviest first over all (stream, head) pairs, so the
    // dispatch order is longest-first across the whole launch and the last
    // round of work-groups holds the shortest tiles; within a tile level the
    // (stream, KV head) group is the fast digit, so with work-group i on XCD
    // i mod 8 the G query heads of a group share an XCD (and its L2) for
    // the whole launch
    const int qt = nqt - 1 - wid / (a.B * a.Hq);
    const int kq = wid % (a.B * a.Hq);
    const int grp = kq % (a.B * a.Hkv), hhq = kq / (a.B * a.Hkv);
    const int b = grp / a.Hkv;
    const int h = (grp % a.Hkv) * a.G + hhq;
    const int g = h / a.G;
    const int tid = threadIdx.x, lane = tid & 63, hf = lane >> 5, l32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int q0 = qt * 128;
    const int row = q0 + 32 * wave + l32;
    const int rc = min(row, a.L - 1);
    const int32_t *kend_b = a.kend + (int64_t)b * a.L;
    const int k_hi = ld_uniform(kend_b, min(q0 + 127, a.L - 1));
    const int kfull = ld_uniform(kend_b, q0);
    const int my_kend = kend_b[rc];
    const int64_t ridx = ((int64_t)b * a.Hq + h) * a.L + rc;
    const float lse2 = a.dl[2 * ridx], Dr = a.dl[2 * ridx + 1];
    const float c2 = a.scale_log2;

    // B fragments of the lane's query row: q and dO, head dims 16 kk + 8 hf + [0, 8)
    bf16x8 qf[KK], dof[KK];
    {
        const uint16_t *qp = a.q + b * a.q_sb + (int64_t)rc * a.q_st + h * a.q_sh + 8 * hf;
        const uint16_t *dp = a.dout + b * a.do_sb + (int64_t)rc * a.do_st + h * a.do_sh + 8 * hf;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            qf[kk] = *(const bf16x8 *)(qp + 16 * kk);
            dof[kk] = *(const bf16x8 *)(dp + 16 * kk);
        }
    }
    const char *kg = (const char *)(a.k + b * a.k_sb + g * a.k_sh);
    const char *vg = (const char *)(a.v + b * a.v_sb + g * a.v_sh);
    const int64_t kst = 2 * a.k_st, vst = 2 * a.v_st;
    auto issue_tile = [&](int t) {
        const uint32_t kl = lds_addr(smem) + (t & 1) * 2 * TILEB;
        dma_rows<D, 4, 64>(kg, kst, t * 64, k_hi - 1, kl, wave, lane);
        dma_rows<D, 4, 64>(vg, vst, t * 64, k_hi - 1, kl + TILEB, wave, lane);
    };
    const uint32_t kbase = (uint32_t)(l32 * ROWB + 16 * (hf ^ swz<D>(l32)));
    uint32_t tb[2];
    tr_bases<D>(lane, tb);

    f32x16 acc[MD];
#pragma unroll
    for (int md = 0; md < MD; ++md)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[md][v] = 0.f;
    const int ntile = (k_hi + 63) / 64;
    if (ntile > 0) issue_tile(0);
    wait_vm_lgkm<0>();
    wg_barrier();
    for (int t = 0; t < ntile; ++t) {
        // the other stage was last read before the previous barrier
        if (t + 1 < ntile) issue_tile(t + 1);
        const char *kt = smem + (t & 1) * 2 * TILEB, *vt = kt + TILEB;
        const bool need_mask = (t + 1) * 64 > kfull;
        // one half of the tile (32 keys) at a time, so that S^T and dP^T of
        // a half, not of the whole tile, are live
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            // S^T = K Q^T and dP^T = V dO^T (keys as rows)
            f32x16 S, dPt;
#pragma unroll
            for (int v = 0; v < 16; ++v) S[v] = dPt[v] = 0.f;
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const bf16x8 ka = *(const bf16x8 *)(kt + mb * 32 * ROWB + (kbase ^ (32 * kk)));
                S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[kk], S, 0, 0, 0);
                const bf16x8 va = *(const bf16x8 *)(vt + mb * 32 * ROWB + (kbase ^ (32 * kk)));
                dPt = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, dof[kk], dPt, 0, 0, 0);
            }
            // dS^T = P^T (dP^T - D), rounded to bf16 as B fragments
            bf16x8 dsf[2];
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int key = t * 64 + mb * 32 + 8 * (v >> 2) + 4 * hf + (v & 3);
                const float p0 = fast_exp2(__builtin_fmaf(S[v], c2, -lse2));
                const float p = (!need_mask || key < my_kend) ? p0 : 0.f;
                dsf[v >> 3][v & 7] = (__bf16)(p * (dPt[v] - Dr));
            }
            // dQ^T += K^T dS^T over this half's keys
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
                for (int md = 0; md < MD; ++md)
                    acc[md] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<D>(kt, tb, 2 * mb + k2, md), dsf[k2],
                                                                     acc[md], 0, 0, 0);
        }
        wait_vm_lgkm<0>();   // tile t + 1 landed (and this tile's LDS reads are done)
        wg_barrier();
    }
    if (row < a.L) {
        float *op = a.dq + b * a.dq_sb + (int64_t)row * a.dq_st + h * a.dq_sh;
#pragma unroll
        for (int md = 0; md < MD; ++md)
#pragma unroll
            for (int gq = 0; gq < 4; ++gq) {
                f32x4 val;
#pragma unroll
                for (int e = 0; e < 4; ++e) val[e] = acc[md][4 * gq + e] * a.scale;
                *(f32x4 *)(op + 32 * md + 8 * gq + 4 * hf) = val;
            }
    }
}

// dK and dV: one work-group = (stream, KV head, 128 keys), 8 waves: wave w
// owns keys 32 (w % 4) .. + 31 and belongs to group w / 4.  The
// work-group's K and V stay in LDS; the chunks of 32 query rows (every row
// that sees any of these keys, for every query head of the KV group, walked
// from the sequence end) alternate between the two groups, each with its own
// two LDS stages, so two waves share every SIMD.  At the end group 1 hands its
// partial sums to group 0 through LDS (fixed order: group 0's + group 1's).
template <int D>
__global__ __launch_bounds__(512) void bwd_dkdv_kernel(const BwdArgs a) {
    constexpr int ROWB = 2 * D, KK = D / 16, MD = D / 32;
    constexpr int TILEK = 128 * ROWB, TILEC = 32 * ROWB;
    constexpr int CPR = ROWB / 16, RPP = 512 / CPR, NPK = 128 / RPP;
    constexpr int SMEM = 2 * TILEK + 2 * 2 * 2 * TILEC;   // K, V; [group][stage][Q, dO]
    static_assert(2 * 4 * MD * 16 * 64 * 4 <= SMEM, "the partial sums fit the tiles' space");
    __shared__ __attribute__((aligned(1024))) char smem[SMEM];
    __shared__ __attribute__((aligned(16))) float sdl[2][2][2][32];   // [group][stage][lse2, D][row]
    __shared__ __attribute__((aligned(16))) int skend[2][2][32];
    const int nkt = (a.L + 127) / 128;
    const int wid = blockIdx.x;
    // Key tiles from the first keys (seen by the most rows: the heaviest)
    // over all (stream, KV head) groups, so the dispatch order is
    // longest-first across the whole launch.  Work-group i runs on XCD
    // i mod 8: when the group count is a multiple of 8, XCD x keeps groups
    // x, x + 8, ... for the whole launch and takes their key tiles in blocks
    // of KB_DKDV, the tiles of a block of one group one after another, so
    // they start together and walk the same rows at about the same time
    // (one L2 read serves them); the launch is rounded up to whole blocks
    // and work-groups past the last key tile exit at once.
    const int ngrp = a.B * a.Hkv;
    int kt, grpi;
    if (ngrp % NUM_XCD == 0) {
        const int gpx = ngrp / NUM_XCD, x = wid % NUM_XCD, l = wid / NUM_XCD;
        const int kb = l / (gpx * KB_DKDV), r = l - kb * gpx * KB_DKDV;
        const int gi = r / KB_DKDV;
        kt = kb * KB_DKDV + (r - gi * KB_DKDV);
        grpi = x + NUM_XCD * gi;
        if (kt >= nkt) return;
    } else {
        kt = wid / ngrp;
        grpi = wid % ngrp;
    }
    const int kvh = grpi % a.Hkv;
    const int b = grpi / a.Hkv;
    const int tid = threadIdx.x, lane = tid & 63, hf = lane >> 5, l32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = wave >> 2, sub = wave & 3, gtid = tid & 255;
    const int kw0 = kt * 128;
    const int key = kw0 + 32 * sub + l32;
    const float c2 = a.scale_log2;
    // the work-group's K and V (rows past the end repeat the last key)
    {
        const int lr = tid / CPR, lc = tid % CPR;
        const uint16_t *kg = a.k + b * a.k_sb + kvh * a.k_sh + 8 * lc;
        const uint16_t *vg = a.v + b * a.v_sb + kvh * a.v_sh + 8 * lc;
#pragma unroll
        for (int p = 0; p < NPK; ++p) {
            const int r = lr + p * RPP;
            const int kr = min(kw0 + r, a.L - 1);
            *(u32x4 *)(smem + tile_off<D>(r, lc)) = *(const u32x4 *)(kg + (int64_t)kr * a.k_st);
            *(u32x4 *)(smem + TILEK + tile_off<D>(r, lc)) = *(const u32x4 *)(vg + (int64_t)kr * a.v_st);
        }
    }
    // first row that sees any of these keys (key ends do not decrease)
    const int32_t *kend_b = a.kend + (int64_t)b * a.L;
    int lo = 0, hi = a.L - 1;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (ld_uniform(kend_b, mid) > kw0) hi = mid; else lo = mid + 1;
    }
    const int i0 = lo;
    // Chunks of 32 query rows counted from the sequence end, down to row i0,
    // with the query heads innermost: chunk it holds rows L - 32 (c + 1) ..
    // L - 32 c - 1 (c = it / G) of head it % G.  The work-groups of a KV head
    // (different key tiles, running side by side) then read the same rows at
    // about the same time and the L2 serves them once.  Rows before i0 see
    // none of these keys, so the masking zeroes their terms.
    const int nch = (a.L - i0 + 31) / 32;
    const int total = a.G * nch;            // chunks; group grp takes chunks grp, grp + 2, ...
    const int nstep = (total + 1) / 2;

    float lreg = 0.f, dreg = 0.f;
    int kreg = 0;
    auto chunk_base = [&](int it) -> uint32_t { return (uint32_t)(2 * TILEK + ((grp * 2 + (it >> 1 & 1)) * 2) * TILEC); };
    // the DMA of chunk it (Q and dO rows) and the (lse2, D, key end) of its
    // rows into registers; group-uniform
    auto issue_chunk = [&](int it) {
        const int c = it / a.G, hh = it - c * a.G;
        const int h = kvh * a.G + hh;
        const int r0 = a.L - 32 * (c + 1);   // may be negative: such rows are no rows
        const uint32_t base = lds_addr(smem) + chunk_base(it);
        dma_rows<D, 4, 32>((const char *)(a.q + b * a.q_sb + h * a.q_sh), 2 * a.q_st, r0, a.L - 1, base, sub, lane);
        dma_rows<D, 4, 32>((const char *)(a.dout + b * a.do_sb + h * a.do_sh), 2 * a.do_st, r0, a.L - 1,
                           base + TILEC, sub, lane);
        if (gtid < 32) {
            const int r = r0 + gtid;
            if (r >= 0) {
                const int64_t idx = ((int64_t)b * a.Hq + h) * a.L + r;
                lreg = a.dl[2 * idx];
                dreg = a.dl[2 * idx + 1];
                kreg = kend_b[r];
            } else {
                lreg = 0.f;
                dreg = 0.f;
                kreg = 0;   // no key visible
            }
        }
    };
    auto store_rowinfo = [&](int it) {
        if (gtid < 32) {
            const int st = it >> 1 & 1;
            sdl[grp][st][0][gtid] = lreg;
            sdl[grp][st][1][gtid] = dreg;
            skend[grp][st][gtid] = kreg;
        }
    };
    const uint32_t kbase = (uint32_t)(l32 * ROWB + 16 * (hf ^ swz<D>(l32)));
    uint32_t tb[2];
    tr_bases<D>(lane, tb);

    f32x16 dk[MD], dv[MD];
#pragma unroll
    for (int md = 0; md < MD; ++md)
#pragma unroll
        for (int v = 0; v < 16; ++v) dk[md][v] = dv[md][v] = 0.f;
    if (grp < total) {
        issue_chunk(grp);
        store_rowinfo(grp);
    }
    wait_vm_lgkm<0>();
    wg_barrier();
    const char *ktile = smem + 32 * sub * ROWB, *vtile = smem + TILEK + 32 * sub * ROWB;
    for (int s = 0; s < nstep; ++s) {
        const int it = 2 * s + grp;          // this group's chunk
        const int nx = it + 2;               // its next one (other stage)
        if (nx < total) issue_chunk(nx);
        if (it < total) {
            const int st = it >> 1 & 1;
            const char *qt = smem + chunk_base(it), *dt = qt + TILEC;
            // S = Q K^T and dP = dO V^T: query rows x this wave's 32 keys
            f32x16 S, dP;
#pragma unroll
            for (int v = 0; v < 16; ++v) S[v] = dP[v] = 0.f;
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const bf16x8 qa = *(const bf16x8 *)(qt + (kbase ^ (32 * kk)));
                const bf16x8 kb = *(const bf16x8 *)(ktile + (kbase ^ (32 * kk)));
                S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, kb, S, 0, 0, 0);
                const bf16x8 da = *(const bf16x8 *)(dt + (kbase ^ (32 * kk)));
                const bf16x8 vb = *(const bf16x8 *)(vtile + (kbase ^ (32 * kk)));
                dP = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da, vb, dP, 0, 0, 0);
            }
            // the lane's 16 query rows 8 (v / 4) + 4 hf + v % 4
            bf16x8 pf[2], dsf[2];
#pragma unroll
            for (int gq = 0; gq < 4; ++gq) {
                const f32x4 l4 = *(const f32x4 *)&sdl[grp][st][0][8 * gq + 4 * hf];
                const f32x4 d4 = *(const f32x4 *)&sdl[grp][st][1][8 * gq + 4 * hf];
                const int4 k4 = *(const int4 *)&skend[grp][st][8 * gq + 4 * hf];
                const int ke[4] = {k4.x, k4.y, k4.z, k4.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int v = 4 * gq + e;
                    const float p0 = fast_exp2(__builtin_fmaf(S[v], c2, -l4[e]));
                    const float p = key < ke[e] ? p0 : 0.f;
                    pf[v >> 3][v & 7] = (__bf16)p;
                    dsf[v >> 3][v & 7] = (__bf16)(p * (dP[v] - d4[e]));
                }
            }
            // dV^T += dO^T P and dK^T += Q^T dS
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                for (int md = 0; md < MD; ++md) {
                    dv[md] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<D>(dt, tb, ks, md), pf[ks], dv[md], 0, 0, 0);
                    dk[md] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<D>(qt, tb, ks, md), dsf[ks], dk[md], 0, 0, 0);
                }
        }
        // the row data of the next chunk goes to the other stage, which was
        // last read before the previous barrier
        if (nx < total) store_rowinfo(nx);
        wait_vm_lgkm<0>();   // the next chunks landed; this step's LDS reads are done
        wg_barrier();
    }
    // group 1 -> LDS -> group 0, in register order (conflict-free)
    float *part = (float *)smem;
    const int pbase = (sub * MD) * 16 * 64 + lane;
    if (grp == 1) {
#pragma unroll
        for (int md = 0; md < MD; ++md)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                part[pbase + (md * 16 + v) * 64] = dk[md][v];
                part[4 * MD * 16 * 64 + pbase + (md * 16 + v) * 64] = dv[md][v];
            }
    }
    wait_vm_lgkm<0>();
    wg_barrier();
    if (grp == 0 && key < a.L) {
        float *kp = a.dk + b * a.dk_sb + (int64_t)key * a.dk_st + kvh * a.dk_sh;
        float *vp = a.dv + b * a.dv_sb + (int64_t)key * a.dv_st + kvh * a.dv_sh;
#pragma unroll
        for (int md = 0; md < MD; ++md)
#pragma unroll
            for (int gq = 0; gq < 4; ++gq) {
                f32x4 kv, vv;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int v = 4 * gq + e;
                    kv[e] = (dk[md][v] + part[pbase + (md * 16 + v) * 64]) * a.scale;
                    vv[e] = dv[md][v] + part[4 * MD * 16 * 64 + pbase + (md * 16 + v) * 64];
                }
                *(f32x4 *)(kp + 32 * md + 8 * gq + 4 * hf) = kv;
                *(f32x4 *)(vp + 32 * md + 8 * gq + 4 * hf) = vv;
            }
    }
}

template <int D>
int launch_bwd_t(const BwdArgs &a, hipStream_t st) {
    const int64_t rows = (int64_t)a.B * a.L * a.Hq;
    const int64_t rpb = 256 / (D / 8);
    hipLaunchKernelGGL(bwd_prep_kernel<D>, dim3((unsigned)((rows + rpb - 1) / rpb)), dim3(256), 0, st, a);
    if (int e = (int)hipGetLastError()) return e;
    const int64_t nqt = (a.L + 127) / 128;
    hipLaunchKernelGGL(bwd_dq_kernel<D>, dim3((unsigned)(a.B * a.Hq * nqt)), dim3(256), 0, st, a);
    if (int e = (int)hipGetLastError()) return e;
    const int64_t ngrp = (int64_t)a.B * a.Hkv;
    const int64_t grid = ngrp % NUM_XCD == 0 ? ngrp * ((nqt + KB_DKDV - 1) / KB_DKDV) * KB_DKDV : ngrp * nqt;
    hipLaunchKernelGGL(bwd_dkdv_kernel<D>, dim3((unsigned)grid), dim3(512), 0, st, a);
    return (int)hipGetLastError();
}

}  // namespace

int launch_prefill_bwd(const BwdArgs &a, int head_dim, void *stream) {
    hipStream_t st = (hipStream_t)stream;
    if (head_dim == 128) return launch_bwd_t<128>(a, st);
    if (head_dim == 64) return launch_bwd_t<64>(a, st);
    return (int)hipErrorInvalidValue;
}

}  // namespace ws
