// gfx950 (CDNA4) kernels of libmtn: plan upload/apply (block-table updates
// and fp64 RoPE angles), fused RoPE + append + evict, vector GQA attention
// over sinks ∪ window (decode, and the fp32 chunk prefill) with a split-K
// log-sum-exp merge, the debug poison kernel and the HBM copy probe.
//
// Method: Metronome (arXiv 2607.02640) §4.1 / App. A -- a query at absolute
// position t attends to keys k <= t with k < S or k in the W positions ending
// at t; sinks are visited first, segments of a split decode are merged once.
#include "mtn_kernels.h"
#include "mtn_device.h"

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>
#include <type_traits>

namespace mtn {
namespace {

// ---------------------------------------------------------------------------
// plan apply: block-table updates + RoPE (cos, sin) table in fp64
// ---------------------------------------------------------------------------
__global__ void k_plan_apply(const int32_t *__restrict__ upd_idx,
                             const int32_t *__restrict__ upd_val, int32_t n_upd,
                             int32_t *__restrict__ table, const int32_t *__restrict__ tok_pos,
                             int32_t n_tok, const double *__restrict__ inv_freq, int32_t half_d,
                             float2 *__restrict__ rope) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n_upd) table[upd_idx[i]] = upd_val[i];
    int64_t total = (int64_t)n_tok * half_d;
    for (int64_t j = i; j < total; j += (int64_t)gridDim.x * blockDim.x) {
        int32_t t = (int32_t)(j / half_d), f = (int32_t)(j % half_d);
        double a = (double)tok_pos[t] * inv_freq[f];
        double sn, cs;
        sincos(a, &sn, &cs);
        rope[j] = make_float2((float)cs, (float)sn);
    }
}

// ---------------------------------------------------------------------------
// fused RoPE + append + evict: one workgroup per (run, kv head), a run being
// one sequence's tokens in consecutive slots of one block
// ---------------------------------------------------------------------------
// Wave w takes the run's tokens w, w + 4, ...; per token, lane i rotates the
// pair (i, i + D/2) and stores both elements into the token's K row
// (consecutive lanes, consecutive bytes) and puts the values into an LDS tile
// [D][16].  After the barrier the V^T tile [D][16] of the block takes, per
// store instruction, 256 consecutive elements of the run's slots
// [off0, off0 + len) in memory order: whole row segments instead of one
// 2-byte element per 32 bytes.
constexpr int kAppendWaves = 4;
template <typename T>
__global__ __launch_bounds__(64 * kAppendWaves) void k_append(PoolGeom g, PlanView p, int32_t layer,
                                                            const T *__restrict__ k,
                                                            const T *__restrict__ v,
                                                            const int32_t *__restrict__ run_tok0,
                                                            const int32_t *__restrict__ run_len) {
    __shared__ T tr[128 * kBlock];  // the run's values, [d][slot]
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int h = (int)(blockIdx.x % g.hkv);
    const int r = (int)(blockIdx.x / g.hkv);
    const int t0 = run_tok0[r], len = run_len[r];
    const int D = g.d, half = D / 2;
    uint8_t *tile = (uint8_t *)g.kv + (int64_t)layer * g.layer_stride +
                    (int64_t)p.tok_block[t0] * g.block_stride + (int64_t)h * g.head_stride;
    T *K = (T *)tile;
    T *VT = (T *)(tile + g.tile_bytes);
    const int off0 = p.tok_off[t0];
#pragma unroll
    for (int jj = 0; jj < kBlock / kAppendWaves; ++jj) {
        const int j = w + kAppendWaves * jj;
        if (j >= len) break;
        const int t = t0 + j;
        const int64_t row = p.tok_row[t];
        const T *kr = k + (row * g.hkv + h) * D;
        const T *vr = v + (row * g.hkv + h) * D;
        T *kd = K + (off0 + j) * D;
        for (int i = lane; i < half; i += 64) {
            const float2 cs = p.rope[(int64_t)t * half + i];
            const float x0 = to_f32(kr[i]), x1 = to_f32(kr[i + half]);
            kd[i] = from_f32<T>(fmaf(x0, cs.x, -x1 * cs.y));
            kd[i + half] = from_f32<T>(fmaf(x1, cs.x, x0 * cs.y));
            tr[i * kBlock + j] = vr[i];
            tr[(i + half) * kBlock + j] = vr[i + half];
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < D * len; e += 64 * kAppendWaves) {
        const int d = e / len, j = e - d * len;
        VT[d * kBlock + off0 + j] = tr[d * kBlock + j];
    }
}

// ---------------------------------------------------------------------------
// vector attention: one wavefront per (query token, kv head, split segment)
// ---------------------------------------------------------------------------
template <typename T, int D>
struct Lay {
    static constexpr int E = (int)sizeof(T);
    static constexpr int NB = D * E / 4;       // bytes per lane of a K (or V^T) tile
    static constexpr int NV4 = NB / 16;        // uint4 loads per lane per tile
    static constexpr int QD = D / 4;           // K dims per lane (one quarter row)
    static constexpr int VD = D / 64;          // V^T rows (dims) per lane
    static constexpr int VW = kBlock * E / 4;  // dwords per V^T row
    static_assert(NB % 16 == 0, "tile slice must be whole uint4s");
};

template <typename T, int D, int G>
struct QRegs;
template <int D, int G>
struct QRegs<bf16_t, D, G> {
    uint32_t v[G][D / 8];  // bf16 pairs of the lane's quarter, pre-scaled
};
template <int D, int G>
struct QRegs<float, D, G> {
    float v[G][D / 4];
};

// Decode launch shape per group size G: WPU waves share each K/V block (a
// wave owns at most 4 of the G heads), NG wave groups split a unit's keys,
// and each group double-buffers its blocks in LDS.  Measured at the
// 128-session G = 8 (Hkv = 4), 64-session G = 1 and 256-session G = 4
// shapes: small rings that let more workgroups stay resident beat deeper
// rings, and two groups per unit where G = 8 put two waves on every SIMD
// (6.1 TB/s vs 5.3 TB/s with one group and a 64 KiB ring).
template <int G>
struct DecodeShape {
#ifdef MTN_DECODE_HEADS_PER_WAVE
    static constexpr int WPU = G >= MTN_DECODE_HEADS_PER_WAVE ? G / MTN_DECODE_HEADS_PER_WAVE : 1;
#else
    static constexpr int WPU = G >= 4 ? G / 4 : 1;
#endif
#ifdef MTN_DECODE_GROUPS
    static constexpr int NG = MTN_DECODE_GROUPS;
#else
    static constexpr int NG = WPU >= 2 ? 2 : 1;
#endif
#ifdef MTN_DECODE_NBUF
    static constexpr int NBUF = MTN_DECODE_NBUF;
#else
    static constexpr int NBUF = 2;
#endif
};

// One work unit = (query token, kv head, split segment), served by one
// workgroup of NG wave groups of WPU waves each.  The unit's keys are cut
// into NG consecutive segments, one per group; each group streams its segment
// through its own ring of K/V^T blocks in LDS (each wave issues 1/WPU of every
// block's DMA) and its waves split the G query heads of the KV group: wave w
// of a group owns heads w*HW .. w*HW + HW - 1, HW = G / WPU <= 4, so every
// lane owns at most one head in the online softmax.  One barrier per block
// step publishes the landed blocks and frees the buffers consumed before
// them.  At the end the groups' (max, sum, acc) are merged through LDS by
// log-sum-exp, so several waves per SIMD stream one unit with no second
// launch.
template <typename T, int D, int G, int WPU, int NG, int NBUF>
__global__ __launch_bounds__(64 * WPU * NG) void k_attn_valu(AttnArgs a) {
    using L = Lay<T, D>;
    constexpr int HW = G / WPU;                     // heads per wave
    static_assert(HW * WPU == G && HW <= 4, "head split");
    static_assert(NBUF >= 2 && NBUF <= 8, "ring depth");
    constexpr int BLK = 2 * kBlock * D * L::E;      // K + V^T bytes of one block (one head)
    constexpr int NCH = BLK / 16;                   // 16-byte chunks per block
    constexpr int NI = NCH / 64;                    // DMA instructions per block
    constexpr int NIW = NI / WPU;                   // ... issued by each wave
    static_assert(NIW * WPU == NI && NIW >= 1, "DMA split");
    static_assert(NG == 1 || NG * G * D * 4 <= NG * NBUF * BLK, "merge scratch fits the ring");
    constexpr int NW = WPU * NG;                    // waves per workgroup
    __shared__ __attribute__((aligned(16))) uint8_t ring[NG][NBUF][BLK];
    __shared__ __attribute__((aligned(16))) float sP[NW][sizeof(T) == 2 ? 1 : 2][HW][kBlock];
    __shared__ float sA[NW][2][HW];
    __shared__ float sM[NW][HW], sL[NW][HW];

    const int lane = threadIdx.x & 63;
    // wave-uniform indices live in scalar registers: the block-table and plan
    // reads below become scalar loads, which do not share the vector-memory
    // counter the LDS ring is synchronised with
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int grp = wv / WPU;                       // wave group (key segment)
    const int wq = wv - grp * WPU;                  // wave inside the group
    const PoolGeom &g = a.g;
    const UnitIdx ui = decode_unit(blockIdx.x, (uint32_t)a.n_split, (uint32_t)g.hkv);
    const int split = ui.split, kvh = ui.kvh, t = ui.t;
    const int sid = __builtin_amdgcn_readfirstlane(a.p.tok_sid[t]);
    const int pos = __builtin_amdgcn_readfirstlane(a.p.tok_pos[t]);
    const int64_t row = __builtin_amdgcn_readfirstlane(a.p.tok_row[t]);
    const int key = lane >> 2, qtr = lane & 3;
    const int h0 = wq * HW;  // first head of this wave inside the KV group
    // Decode with a fused append: the group holding the unit's last segment
    // (it always ends at the query's own position, the newest key) takes that
    // key from the inputs instead of the pool -- masking its slot out of the
    // ring scan -- and writes the key and value into the pool at the end, for
    // later launches.  No wave of this launch reads that slot as a key.
    const bool own_new = a.k_new != nullptr && split == a.n_split - 1 && grp == NG - 1;

    // ---- work range and the first prefetches (issued before the q prologue)
    // segment seg = split * NG + grp of nseg = n_split * NG covers virtual
    // blocks [v0, v1); sinks sit in virtual block 0, so only segment 0 reads them
    const VisRange vr = vis_range(g, pos);
    const int nv = vr.n_sb + vr.n_rb;
    const uint32_t nseg = (uint32_t)a.n_split * NG;
    const uint32_t seg = (uint32_t)split * NG + grp;
    const int v0 = __builtin_amdgcn_readfirstlane(seg_begin(seg, nseg, nv));
    const int v1 = __builtin_amdgcn_readfirstlane(seg_begin(seg + 1, nseg, nv));
    const int nblk = v1 - v0;
    // the barrier is workgroup-wide: every group runs the longest group's steps
    int nstep = 0;
    {
        int b = seg_begin((uint32_t)split * NG, nseg, nv);
#pragma unroll
        for (int q2 = 0; q2 < NG; ++q2) {
            const int e = seg_begin((uint32_t)split * NG + q2 + 1, nseg, nv);
            nstep = max(nstep, e - b);
            b = e;
        }
    }
    nstep = __builtin_amdgcn_readfirstlane(nstep);
    const uint8_t *head_base = g.kv + (int64_t)a.layer * g.layer_stride + (int64_t)kvh * g.head_stride;
    const int32_t *trow = g.table + (int64_t)sid * g.row_len;
    const uint32_t ring0 = lds_addr(&ring[grp][0][0]);

    BlockIter it_issue(g, vr, v0), it_proc(g, vr, v0);
    auto issue = [&](int i) {  // next block of the range -> ring slot i % NBUF (this wave's share)
        int lb, lo, hi;
        it_issue.get(&lb, &lo, &hi);
        it_issue.next();
        int phys = scalar_ld(trow, __builtin_amdgcn_readfirstlane(lb));
        phys = phys < 0 ? 0 : phys;
        const uint8_t *src = head_base + (int64_t)phys * g.block_stride;
        const uint32_t dst = ring0 + (uint32_t)((i % NBUF) * BLK);
#pragma unroll
        for (int jj = 0; jj < NIW; ++jj) {
            const int j = wq * NIW + jj;
            dma16(src + swz(j * 64 + lane) * 16, dst + j * 1024);
        }
    };
    const int pre = nblk < NBUF - 1 ? nblk : NBUF - 1;
    for (int i = 0; i < pre; ++i) issue(i);

    // fused append: this lane's value dims of the newest key (set in the q
    // prologue by the owning group)
    float v_new[L::VD];
#pragma unroll
    for (int r = 0; r < L::VD; ++r) v_new[r] = 0.f;

    // ---- q prologue: rotate at pos, fold the softmax scale (log2 domain).
    // With a fused append, the owning group also rotates the newest key's
    // quarter with the same RoPE values, exactly as the append kernel does
    // (fp32, then rounded to the stored type), and accumulates its scores for
    // this wave's heads as the q pairs come out.  The pool copy is written
    // after the ring loop (nothing in this launch reads it, and no ring wait
    // then covers the stores).
    QRegs<T, D, HW> q;
    uint32_t knew[(D / 4) * sizeof(T) / 4];  // the rotated key quarter, stored layout
    {
        // each lane reads its quarter and the RoPE partner quarter of every
        // head as whole 16-byte vectors
        const T *qb = (const T *)a.q + (row * g.hq + (int64_t)kvh * G + h0) * D;
        const float2 *rp = a.p.rope + (int64_t)t * (D / 2) + (qtr & 1) * L::QD;
        const int d0 = qtr * L::QD;
        const int dp = (qtr ^ 2) * L::QD;
        const float sgn = (qtr < 2) ? -1.f : 1.f;
        constexpr int EPV = 16 / L::E;        // elements per 16-byte vector
        constexpr int NVQ = L::QD / EPV;      // vectors per quarter
        const T *kb = own_new ? (const T *)a.k_new + (row * g.hkv + kvh) * D : nullptr;
        // element pairs of a 16-byte vector: (lo, hi) floats of dword e/2
        auto unpack = [](const uint4 &v, float *x) {
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < EPV; ++e) {
                if constexpr (sizeof(T) == 2)
                    x[e] = __uint_as_float((e & 1) ? (w[e / 2] & 0xFFFF0000u) : (w[e / 2] << 16));
                else
                    x[e] = __uint_as_float(w[e]);
            }
        };
#pragma unroll
        for (int vq = 0; vq < NVQ; ++vq) {
            float2 cs[EPV];
#pragma unroll
            for (int e = 0; e < EPV; ++e) cs[e] = rp[vq * EPV + e];
            uint32_t kv4[4];  // the newest key's rotated vector (stored layout)
            if (own_new) {
                float xs[EPV], ys[EPV];
                unpack(((const uint4 *)(kb + d0))[vq], xs);
                unpack(((const uint4 *)(kb + dp))[vq], ys);
#pragma unroll
                for (int e = 0; e < EPV; e += 2) {
                    const float k0 = fmaf(xs[e], cs[e].x, sgn * ys[e] * cs[e].y);
                    const float k1 = fmaf(xs[e + 1], cs[e + 1].x, sgn * ys[e + 1] * cs[e + 1].y);
                    if constexpr (sizeof(T) == 2) {
                        kv4[e / 2] = pack_bf16x2(k0, k1);
                    } else {
                        kv4[e] = __float_as_uint(k0);
                        kv4[e + 1] = __float_as_uint(k1);
                    }
                }
#pragma unroll
                for (int c = 0; c < 4; ++c) knew[vq * 4 + c] = kv4[c];
            }
#pragma unroll
            for (int h = 0; h < HW; ++h) {
                float xs[EPV], ys[EPV];
                unpack(((const uint4 *)(qb + (int64_t)h * D + d0))[vq], xs);
                unpack(((const uint4 *)(qb + (int64_t)h * D + dp))[vq], ys);
#pragma unroll
                for (int e = 0; e < EPV; e += 2) {
                    const int i = vq * EPV + e;
                    const float r0 = fmaf(xs[e], cs[e].x, sgn * ys[e] * cs[e].y) * a.scale_log2;
                    const float r1 = fmaf(xs[e + 1], cs[e + 1].x, sgn * ys[e + 1] * cs[e + 1].y) * a.scale_log2;
                    if constexpr (sizeof(T) == 2) {
                        q.v[h][i / 2] = pack_bf16x2(r0, r1);
                    } else {
                        q.v[h][i] = r0;
                        q.v[h][i + 1] = r1;
                    }
                }
            }
        }
        if (own_new) {
            const T *vb = (const T *)a.v_new + (row * g.hkv + kvh) * D;
#pragma unroll
            for (int r = 0; r < L::VD; ++r) v_new[r] = to_f32(vb[lane * L::VD + r]);
        }
    }

    // the head this lane owns in the softmax (lanes with qtr >= HW duplicate)
    const int hown = qtr < HW ? qtr : qtr % HW;

    float m = -INFINITY, lsum = 0.f;
    float acc[HW][L::VD];
#pragma unroll
    for (int h = 0; h < HW; ++h)
#pragma unroll
        for (int r = 0; r < L::VD; ++r) acc[h][r] = 0.f;

    for (int i = 0; i < nstep; ++i) {
        // this wave's share of block i has landed once at most the shares of
        // the blocks issued after it are outstanding; the barrier then covers
        // the other waves' shares and frees the buffer of block i - 1
        if (i < nblk) vm_wait_blocks<NIW, NBUF - 2>(min(NBUF - 2, nblk - 1 - i));
        if constexpr (NW > 1) __syncthreads();
        if (i >= nblk) continue;  // a shorter segment idles through the last step
        if (i + NBUF - 1 < nblk) issue(i + NBUF - 1);
        const uint8_t *blk = &ring[grp][i % NBUF][0];
        const int buf = i & 1;
        int lb, lo, hi;
        it_proc.get(&lb, &lo, &hi);
        it_proc.next();
        if (scalar_ld(trow, __builtin_amdgcn_readfirstlane(lb)) < 0) hi = lo;  // unassigned: nothing visible
        if (own_new && i == nblk - 1 && hi > lo) --hi;  // the newest key comes from registers

        // QK: this lane's quarter of key `key`, then the quad all-reduce
        uint32_t kw[L::NV4 * 4];
#pragma unroll
        for (int c = 0; c < L::NV4; ++c) {
            uint4 x = *(const uint4 *)(blk + swz(L::NV4 * lane + c) * 16);
            kw[4 * c] = x.x; kw[4 * c + 1] = x.y; kw[4 * c + 2] = x.z; kw[4 * c + 3] = x.w;
        }
        // V^T slice read early: independent of the softmax
        uint32_t vv[L::VD][L::VW];
#pragma unroll
        for (int c = 0; c < L::NV4; ++c) {
            uint4 x = *(const uint4 *)(blk + swz(NCH / 2 + L::NV4 * lane + c) * 16);
            uint32_t *f = &vv[0][0];
            f[4 * c] = x.x; f[4 * c + 1] = x.y; f[4 * c + 2] = x.z; f[4 * c + 3] = x.w;
        }
        // heads innermost: HW independent accumulation chains interleave
        float sc[HW];
#pragma unroll
        for (int h = 0; h < HW; ++h) sc[h] = 0.f;
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int c = 0; c < D / 8; ++c)
#pragma unroll
                for (int h = 0; h < HW; ++h) sc[h] = dot2_bf16(q.v[h][c], kw[c], sc[h]);
        } else {
#pragma unroll
            for (int c = 0; c < D / 4; ++c)
#pragma unroll
                for (int h = 0; h < HW; ++h) sc[h] = fmaf(q.v[h][c], __uint_as_float(kw[c]), sc[h]);
        }
#pragma unroll
        for (int h = 0; h < HW; ++h) sc[h] += dpp<kQuadXor1>(sc[h]);
#pragma unroll
        for (int h = 0; h < HW; ++h) sc[h] += dpp<kQuadXor2>(sc[h]);
        // online softmax of the owned head
        const bool valid = key >= lo && key < hi;
        float s = sc[0];
#pragma unroll
        for (int c = 1; c < HW; ++c) s = (hown == c) ? sc[c] : s;
        s = valid ? s : -INFINITY;
        const float mx = keys_max(s);
        const float m_new = fmaxf(m, mx);
        const float mn = (m_new == -INFINITY) ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m - mn);
        const float p = __builtin_amdgcn_exp2f(s - mn);
        lsum = lsum * alpha + p;
        m = m_new;
        if (lo > 0 || hi < kBlock) {  // zero values of invisible slots (may be NaN)
#pragma unroll
            for (int c = 0; c < L::VW; ++c) {
                uint32_t mask;
                if constexpr (sizeof(T) == 2) {
                    int k0 = 2 * c, k1 = 2 * c + 1;
                    mask = ((k0 >= lo && k0 < hi) ? 0x0000FFFFu : 0u) |
                           ((k1 >= lo && k1 < hi) ? 0xFFFF0000u : 0u);
                } else {
                    mask = (c >= lo && c < hi) ? 0xFFFFFFFFu : 0u;
                }
#pragma unroll
                for (int r = 0; r < L::VD; ++r) vv[r][c] &= mask;
            }
        }
        if constexpr (sizeof(T) == 2) {
            // P and alpha reach the PV lanes through scalar registers: the lane
            // of key 2c+1 packs (p[2c], p[2c+1]) (DPP row shift by one key),
            // readlane broadcasts it, and dot2 takes it as a scalar operand
            const float p_prev = dpp<kRowShr4>(p);
            const uint32_t packed = pack_bf16x2(p_prev, p);
            uint32_t pp[HW][kBlock / 2];
            float al[HW];
#pragma unroll
            for (int h = 0; h < HW; ++h) {
                al[h] = __builtin_bit_cast(float,
                                           __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha), h));
#pragma unroll
                for (int c = 0; c < kBlock / 2; ++c)
                    pp[h][c] = (uint32_t)__builtin_amdgcn_readlane((int)packed, 8 * c + 4 + h);
            }
#pragma unroll
            for (int h = 0; h < HW; ++h)
#pragma unroll
                for (int r = 0; r < L::VD; ++r) acc[h][r] *= al[h];
#pragma unroll
            for (int c = 0; c < kBlock / 2; ++c)
#pragma unroll
                for (int h = 0; h < HW; ++h)
#pragma unroll
                    for (int r = 0; r < L::VD; ++r) acc[h][r] = dot2_bf16(pp[h][c], vv[r][c], acc[h][r]);
        } else {
            if (qtr < HW) {
                sP[wv][buf][qtr][key] = p;
                if (key == 0) sA[wv][buf][qtr] = alpha;
            }
            wave_sync();
#pragma unroll
            for (int h = 0; h < HW; ++h) {
                const float al = sA[wv][buf][h];
#pragma unroll
                for (int r = 0; r < L::VD; ++r) acc[h][r] *= al;
            }
#pragma unroll
            for (int c = 0; c < kBlock; ++c)
#pragma unroll
                for (int h = 0; h < HW; ++h) {
                    const float pc = sP[wv][buf][h][c];
#pragma unroll
                    for (int r = 0; r < L::VD; ++r) acc[h][r] = fmaf(pc, __uint_as_float(vv[r][c]), acc[h][r]);
                }
        }
    }

    if (own_new) {
        // ---- the newest key (rotated in the prologue): its score for the
        // owned head, then one more online-softmax step
        float sn[HW];
#pragma unroll
        for (int h = 0; h < HW; ++h) sn[h] = 0.f;
        constexpr int KW = (int)(sizeof(knew) / 4);
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int c = 0; c < KW; ++c)
#pragma unroll
                for (int h = 0; h < HW; ++h) sn[h] = dot2_bf16(q.v[h][c], knew[c], sn[h]);
        } else {
#pragma unroll
            for (int c = 0; c < KW; ++c)
#pragma unroll
                for (int h = 0; h < HW; ++h) sn[h] = fmaf(q.v[h][c], __uint_as_float(knew[c]), sn[h]);
        }
#pragma unroll
        for (int h = 0; h < HW; ++h) sn[h] += dpp<kQuadXor1>(sn[h]);
#pragma unroll
        for (int h = 0; h < HW; ++h) sn[h] += dpp<kQuadXor2>(sn[h]);
        float s_new = sn[0];
#pragma unroll
        for (int c = 1; c < HW; ++c) s_new = (hown == c) ? sn[c] : s_new;
        const float m_new = fmaxf(m, s_new);  // s_new is finite
        const float alpha = __builtin_amdgcn_exp2f(m - m_new);
        const float pn = __builtin_amdgcn_exp2f(s_new - m_new);
        lsum = lsum * alpha + (key == 0 ? pn : 0.f);
        m = m_new;
#pragma unroll
        for (int h = 0; h < HW; ++h) {
            // lane h holds head h's softmax state (key 0, quarter h)
            const float al = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha), h));
            float ph = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, pn), h));
            if constexpr (sizeof(T) == 2) ph = to_f32(from_f32<bf16_t>(ph));  // as the PV operand
#pragma unroll
            for (int r = 0; r < L::VD; ++r) acc[h][r] = fmaf(ph, v_new[r], acc[h][r] * al);
        }
    }

    // the pool copy of the newest key and value, for later launches: lanes
    // 0..3 write the four quarters of the key row, every lane its value dims
    // (the V^T column).  Issued after the wave's last barrier -- a barrier's
    // release fence would wait for these scattered stores.
    auto store_new = [&]() {
        const int64_t tb = __builtin_amdgcn_readfirstlane(a.p.tok_block[t]);
        const int toff = __builtin_amdgcn_readfirstlane(a.p.tok_off[t]);
        uint8_t *ktile = (uint8_t *)g.kv + (int64_t)a.layer * g.layer_stride + tb * g.block_stride +
                         (int64_t)kvh * g.head_stride;
        if (key == 0) {
            uint4 *kd = (uint4 *)(ktile + ((int64_t)toff * D + qtr * L::QD) * L::E);
#pragma unroll
            for (int c = 0; c < (int)(sizeof(knew) / 16); ++c)
                kd[c] = make_uint4(knew[4 * c], knew[4 * c + 1], knew[4 * c + 2], knew[4 * c + 3]);
        }
        T *VTp = (T *)(ktile + g.tile_bytes);
#pragma unroll
        for (int r = 0; r < L::VD; ++r)
            VTp[(lane * L::VD + r) * kBlock + toff] = from_f32<T>(v_new[r]);
    };

    // ---- finish: reduce the per-lane partial sums, publish (m, l) per head
    {
        const float lt = keys_sum(lsum);
        if (qtr < HW && key == 0) {
            sM[wv][qtr] = m;
            sL[wv][qtr] = lt;
        }
    }
    if constexpr (NG > 1) {
        // groups 1.. hand (m, l, acc) to group 0 through the (drained) ring
        float *scr = (float *)&ring[0][0][0];  // [NG][G][D]
        __syncthreads();
        if (grp > 0) {
#pragma unroll
            for (int h = 0; h < HW; ++h)
#pragma unroll
                for (int r = 0; r < L::VD; ++r)
                    scr[((int64_t)grp * G + h0 + h) * D + lane * L::VD + r] = acc[h][r];
        }
        __syncthreads();
        if (grp > 0) {
            if (own_new && wq == 0) store_new();
            return;
        }
#pragma unroll
        for (int h = 0; h < HW; ++h) {
            float M = sM[wq][h];
#pragma unroll
            for (int q2 = 1; q2 < NG; ++q2) M = fmaxf(M, sM[q2 * WPU + wq][h]);
            const float Mn = (M == -INFINITY) ? 0.f : M;
            float w0 = __builtin_amdgcn_exp2f(sM[wq][h] - Mn);
            float Ls = sL[wq][h] * w0;
#pragma unroll
            for (int r = 0; r < L::VD; ++r) acc[h][r] *= w0;
#pragma unroll
            for (int q2 = 1; q2 < NG; ++q2) {
                const float wg = __builtin_amdgcn_exp2f(sM[q2 * WPU + wq][h] - Mn);
                Ls += sL[q2 * WPU + wq][h] * wg;
#pragma unroll
                for (int r = 0; r < L::VD; ++r)
                    acc[h][r] = fmaf(wg, scr[((int64_t)q2 * G + h0 + h) * D + lane * L::VD + r], acc[h][r]);
            }
            // only group 0's waves read these from here on
            if (lane == 0) {
                sM[wv][h] = M;
                sL[wv][h] = Ls;
            }
        }
    }
    wave_sync();
    const int hq0 = kvh * G + h0;
    if (a.n_split == 1) {
        T *ob = (T *)a.out + (row * g.hq + hq0) * D;
#pragma unroll
        for (int h = 0; h < HW; ++h) {
            const float inv = 1.f / sL[wv][h];
#pragma unroll
            for (int r = 0; r < L::VD; ++r) ob[(int64_t)h * D + lane * L::VD + r] = from_f32<T>(acc[h][r] * inv);
        }
        if (a.lse && lane < HW)
            a.lse[row * g.hq + hq0 + lane] =
                (sM[wv][lane] + __builtin_amdgcn_logf(sL[wv][lane])) * 0.6931471805599453f;
    } else {
        const int64_t ns = a.n_split;
        float *pacc = a.part;
        float *pml = a.part + (int64_t)a.p.n_tok * g.hq * ns * D;
#pragma unroll
        for (int h = 0; h < HW; ++h) {
            int64_t base = (((int64_t)t * g.hq + hq0 + h) * ns + split);
#pragma unroll
            for (int r = 0; r < L::VD; ++r) pacc[base * D + lane * L::VD + r] = acc[h][r];
        }
        if (lane < HW) {
            int64_t base = (((int64_t)t * g.hq + hq0 + lane) * ns + split);
            pml[base * 2] = sM[wv][lane];
            pml[base * 2 + 1] = sL[wv][lane];
        }
    }
    if constexpr (NG == 1) {
        if (own_new && wq == 0) store_new();  // one group: it owns the newest key
    }
}

// Split partials of mtn_attend_decode_noalloc: a file-scope device array, so
// that callers that cannot allocate (graph capture, allocation-free serving
// loops) still have a workspace.  Each GPU holds its own copy for the life of
// the process; every call on one GPU shares it.
constexpr size_t kScratchFloats = (size_t)4 << 20;  // 16 MiB
static __device__ __align__(256) float scratch[kScratchFloats];

// merge split partials: one wave per (token, q head).  Lane s takes split s's
// (max, sum); the splits' accumulators do not depend on them and are loaded in
// the same round, eight splits at a time.  The maximum and the weighted sum
// are formed across the wave, and each split's weight is broadcast from its
// lane.  (One memory round trip for up to eight splits, where a loop over the
// splits first for the maximum and then for the sums took two.)
template <typename T, int D>
__global__ __launch_bounds__(64) void k_merge(AttnArgs a) {
    constexpr int VD = D / 64;  // output dims per lane
    constexpr int CH = 8;       // splits whose accumulators are in flight together
    const int64_t th = blockIdx.x;  // t * Hq + hq
    const int lane = threadIdx.x;
    const int ns = a.n_split;       // 2 .. 64
    const float *pacc = a.part + th * ns * D + lane * VD;
    const float *pml = a.part + (int64_t)a.p.n_tok * a.g.hq * ns * D + th * ns * 2;
    float acc[VD];
#pragma unroll
    for (int r = 0; r < VD; ++r) acc[r] = 0.f;
    float part[CH][VD];
    auto load = [&](int s0) {
#pragma unroll
        for (int c = 0; c < CH; ++c)
#pragma unroll
            for (int r = 0; r < VD; ++r) part[c][r] = pacc[min(s0 + c, ns - 1) * D + r];  // past ns: unused
    };
    load(0);
    const float2 ml0 = *(const float2 *)(pml + 2 * min(lane, ns - 1));  // lanes past ns: unused
    __builtin_amdgcn_sched_barrier(0);  // every load above is in flight before the first wait
    const float2 ml = lane < ns ? ml0 : make_float2(-INFINITY, 0.f);
    float M = ml.x;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) M = fmaxf(M, __shfl_xor(M, m, 64));
    const float Mn = M == -INFINITY ? 0.f : M;
    const float w = ml.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml.x - Mn);
    float Lsum = ml.y * w;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) Lsum += __shfl_xor(Lsum, m, 64);
    for (int s0 = 0; s0 < ns; s0 += CH) {
        if (s0) load(s0);
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            // no branch: a split past ns weighs 0 (its slot repeats a finite partial)
            const float wl = __builtin_bit_cast(
                float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, w), min(s0 + c, 63)));
            const float ws = s0 + c < ns ? wl : 0.f;
#pragma unroll
            for (int r = 0; r < VD; ++r) acc[r] = fmaf(ws, part[c][r], acc[r]);
        }
    }
    const int t = (int)(th / a.g.hq), hq = (int)(th % a.g.hq);
    const int64_t row = a.p.tok_row[t];
    T *ob = (T *)a.out + (row * a.g.hq + hq) * D;
    const float inv = 1.f / Lsum;
#pragma unroll
    for (int r = 0; r < VD; ++r) ob[lane * VD + r] = from_f32<T>(acc[r] * inv);
    if (a.lse && lane == 0)
        a.lse[row * a.g.hq + hq] = (M + __builtin_amdgcn_logf(Lsum)) * 0.6931471805599453f;
}

// ---------------------------------------------------------------------------
// debug poison: NaN into every slot whose live bit is clear
// ---------------------------------------------------------------------------
template <typename T>
__global__ void k_poison(PoolGeom g, int32_t n_layers, int64_t n_blocks,
                         const uint16_t *__restrict__ live) {
    const int64_t n_items = (int64_t)n_layers * n_blocks * g.hkv;
    T nan_v;
    if constexpr (sizeof(T) == 2) nan_v = __builtin_bit_cast(T, (uint16_t)0x7FC0);
    else nan_v = __builtin_bit_cast(T, 0x7FC00000u);
    for (int64_t it = blockIdx.x; it < n_items; it += gridDim.x) {
        int h = (int)(it % g.hkv);
        int64_t b = (it / g.hkv) % n_blocks;
        int l = (int)(it / ((int64_t)g.hkv * n_blocks));
        uint16_t lm = live[b];
        if (lm == 0xFFFF) continue;
        uint8_t *tile = (uint8_t *)g.kv + (int64_t)l * g.layer_stride + b * g.block_stride +
                        (int64_t)h * g.head_stride;
        T *K = (T *)tile;
        T *VT = (T *)(tile + g.tile_bytes);
        for (int e = threadIdx.x; e < kBlock * g.d; e += blockDim.x) {
            int off = e / g.d, d = e % g.d;
            if (!((lm >> off) & 1)) {
                K[e] = nan_v;
                VT[d * kBlock + off] = nan_v;
            }
        }
    }
}

// plain streaming copy, four 16-byte loads in flight per thread
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
__global__ void k_copy(const u32x4_t *__restrict__ src, u32x4_t *__restrict__ dst, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (; i + 3 * stride < n; i += 4 * stride) {
        u32x4_t a = __builtin_nontemporal_load(src + i);
        u32x4_t b = __builtin_nontemporal_load(src + i + stride);
        u32x4_t c = __builtin_nontemporal_load(src + i + 2 * stride);
        u32x4_t d = __builtin_nontemporal_load(src + i + 3 * stride);
        __builtin_nontemporal_store(a, dst + i);
        __builtin_nontemporal_store(b, dst + i + stride);
        __builtin_nontemporal_store(c, dst + i + 2 * stride);
        __builtin_nontemporal_store(d, dst + i + 3 * stride);
    }
    for (; i < n; i += stride) dst[i] = src[i];
}

// streaming read (the achievable read bandwidth of the decode's copy
// mechanism): every wave streams 8 KiB chunks into its own two-slot LDS ring
// with the same non-temporal LDS DMA as the decode, at most two chunks in
// flight, chunks interleaved over the waves; nothing is computed or written
// (`out` is kept for the interface)
constexpr int kReadWaves = 4;
__global__ __launch_bounds__(64 * kReadWaves) void k_read(const uint8_t *__restrict__ src,
                                                        int64_t n_chunks, uint32_t *out) {
    __shared__ __attribute__((aligned(16))) uint8_t ring[kReadWaves][2][8192];
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t gw = (int64_t)blockIdx.x * kReadWaves + w;
    const int64_t tw = (int64_t)gridDim.x * kReadWaves;
    const uint32_t slot0 = lds_addr(&ring[w][0][0]);
    int i = 0;
    for (int64_t c = gw; c < n_chunks; c += tw, ++i) {
        vm_wait<8>();  // the chunk issued two turns ago (this slot's) has landed
        const uint8_t *g = src + c * 8192 + lane * 16;
        const uint32_t dst = slot0 + (uint32_t)((i & 1) * 8192);
#pragma unroll
        for (int j = 0; j < 8; ++j) dma16(g + j * 1024, dst + j * 1024);
    }
    vm_wait<0>();  // no copy may land after the workgroup ends
    (void)out;
}

// ---------------------------------------------------------------------------
// MFMA chunk prefill (bf16 or fp8 pool, D = 128): one workgroup per
// (sequence, row pass, kv head)
// ---------------------------------------------------------------------------
// Rows of the chunk are (token j, group head g) -> r = j * G + g, in tiles of
// 16.  Keys stream in stages of 32 (two 16-token blocks) through LDS.
//   S^T[key][row] = K[key][:] . Qrot[row][:]      (A = K, B = Q^T)
//   O^T[d][row]  += V^T[d][key] . P^T[key][row]   (A = V^T, B = P^T)
// With the 16x16x32 MFMA output layout, lane l holds column (row) l % 16 of
// both S^T and O^T, so a row's softmax state and its accumulators share a
// lane.  The QK product of a stage is two MFMAs per 32-wide slice of d whose
// A rows are permuted keys: row i of MFMA mf holds stage key
// 8 (i / 4) + 4 mf + i % 4.  Lane l (g = l / 16) then holds the scores of the
// eight consecutive stage keys 8g .. 8g + 7, all in block g / 2, which are
// exactly the k slots 8g .. 8g + 7 of its PV B operand; the matching V^T
// A operand is one aligned 16-byte chunk per lane.

#ifndef MTN_PF_WAVES
#define MTN_PF_WAVES 8
#endif
#ifndef MTN_PF_TILES_PER_WAVE
#define MTN_PF_TILES_PER_WAVE 2
#endif
#ifndef MTN_PF_STAGES
#define MTN_PF_STAGES 8
#endif
#ifndef MTN_PF_DMA_WAVES
#define MTN_PF_DMA_WAVES 2
#endif
constexpr int kPfWaves = MTN_PF_WAVES;          // waves per workgroup
constexpr int kPfTpw = MTN_PF_TILES_PER_WAVE;   // 16-row query tiles per wave per pass
constexpr int kPfRowsPerPass = kPfWaves * kPfTpw * 16;
constexpr int kPfStages = MTN_PF_STAGES;        // LDS ring depth in stages of two blocks (16 KiB each)
#ifndef MTN_PF_EARLY
#define MTN_PF_EARLY 3
#endif
constexpr int kPfEarly = MTN_PF_EARLY;          // ring stages copied before the query rotation
constexpr int kPfStageBytes = 16384;

struct PfArgs {
    AttnArgs a;
    const int32_t *items;      // kPfItem-int records, one per (sequence, row pass)
    const uint8_t *zero_page;  // 16 KiB of zeros: the DMA source of absent blocks
    int32_t pass_rows;         // query rows per pass: 128 or kPfRowsPerPass
};

// LDS layout of one stage: K tiles of blocks 0, 1 (the 16-byte chunks of a
// key row permuted by kswz(b, key)), then V^T tiles (the two 16-byte halves of
// a d row swapped on bit 2 of d).  A K read instruction has lanes 0..15 on
// keys {0..3, 8..11} (or {4..7, 12..15}) of both blocks; kswz gives those 16
// (block, key) pairs 16 distinct chunk positions and ignores key bit 2, so
// the second MFMA's rows sit exactly 4 rows (1 KiB) further.  Both patterns
// read at the full LDS rate (measured: 228 and 240 B/clk/CU against 178 for
// a swizzle without the block bit).
__device__ __forceinline__ int kswz(int b, int key) {
    return (key & 3) | ((key & 8) >> 1) | (b << 3);
}
__device__ __forceinline__ int lds_k(int b, int key, int chunk16) {
    return b * 4096 + key * 256 + ((chunk16 ^ kswz(b, key)) << 4);
}
__device__ __forceinline__ int lds_v16(int b, int d, int half) {
    return 8192 + b * 4096 + d * 32 + ((half ^ ((d >> 2) & 1)) << 4);
}
// Byte offset, inside a block's 8 KiB (K tile, V^T tile) pair, of the 16-byte
// chunk that lands at stage byte offset `off`; *b = which block of the stage.
__device__ __forceinline__ int stage_src(int off, int *b) {
    if (off < 8192) {
        *b = off >> 12;
        const int r = off & 4095, key = r >> 8, pos = (r >> 4) & 15;
        return key * 256 + ((pos ^ kswz(*b, key)) << 4);
    }
    const int o2 = off - 8192;
    *b = o2 >> 12;
    const int r = o2 & 4095, d = r >> 5, pos = (r >> 4) & 1;
    return 4096 + d * 32 + ((pos ^ ((d >> 2) & 1)) << 4);
}

// A virtual block of a chunk's key union (sinks first, then the ring run):
// logical block, valid slots [lo, hi), absolute position of slot 0.
struct PfBlock {
    int lb, lo, hi, p0;
    bool sink;
};

// An fp8 stage as the DMA lands it (two block regions of kF8Read bytes: K
// codes, V codes in key quads, exponents) -> the bf16 stage layout above, each
// value code * 2^e exactly.  512 threads: thread tid converts, in block
// tid >> 8, K dims 8 (tid & 15) .. + 7 of key (tid >> 4) & 15, and V dims
// 2 (tid & 63), 2 (tid & 63) + 1 of keys 4 ((tid >> 6) & 3) .. + 3.
__device__ __forceinline__ void f8_stage_to_bf16(const uint8_t *src, uint8_t *dst, int tid) {
    const int b = tid >> 8;
    const uint8_t *blk = src + b * kF8Read;
    {
        const int key = (tid >> 4) & 15, hc = tid & 15;
        const uint2 c = *(const uint2 *)(blk + key * kF8D + hc * 8);
        // one scale for the whole row: the scaling conversion multiplies both
        // codes of a pair by the key's 2^e, exactly
        const float sk = __uint_as_float((uint32_t)blk[kF8Exp + key] << 23);
        auto cv = [&](uint32_t w, auto hi) {
            return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(
                                                    w, sk, decltype(hi)::value));
        };
        *(uint4 *)(dst + lds_k(b, key, hc)) =
            make_uint4(cv(c.x, std::false_type{}), cv(c.x, std::true_type{}),
                       cv(c.y, std::false_type{}), cv(c.y, std::true_type{}));
    }
    {
        const int kg = (tid >> 6) & 3, dp = tid & 63;
        const uint2 c = *(const uint2 *)(blk + kF8Tile + (kg * kF8D + 2 * dp) * 4);
        const uint32_t ew = *(const uint32_t *)(blk + kF8Exp + kBlock + 4 * kg);
        float sv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) sv[r] = __uint_as_float(((ew >> (8 * r)) & 0xFFu) << 23);
        const uint32_t w[2] = {c.x, c.y};
#pragma unroll
        for (int x = 0; x < 2; ++x) {  // dim 2 dp + x: keys 4 kg .. 4 kg + 3
            const auto lo = __builtin_amdgcn_cvt_pk_f32_fp8(w[x], false);
            const auto hi = __builtin_amdgcn_cvt_pk_f32_fp8(w[x], true);
            *(uint2 *)(dst + lds_v16(b, 2 * dp + x, kg >> 1) + (kg & 1) * 8) =
                make_uint2(pack_bf16x2(lo[0] * sv[0], lo[1] * sv[1]),
                           pack_bf16x2(hi[0] * sv[2], hi[1] * sv[3]));
        }
    }
}

// F8: the pool holds E4M3 codes.  Each stage then lands as two kF8Read-byte
// regions (per block four 1 KiB DMA instructions plus the 32 exponent
// bytes), and every stage is converted into one of two bf16 stage buffers (a
// second barrier) before the same MFMA stage body runs on it.
template <int G, bool F8>
__global__ __launch_bounds__(64 * kPfWaves) void k_prefill_mfma(PfArgs pa) {
    constexpr int D = 128;
    constexpr int SB = F8 ? 2 * kF8Read : kPfStageBytes;  // bytes of a ring stage
    static_assert(kPfStages >= 3 && kPfStages <= 8, "ring depth (the DMA waits count at most 63)");
    static_assert(kPfEarly >= 1 && kPfEarly <= kPfStages - 1, "early stages are ring prologue stages");
    __shared__ __attribute__((aligned(16))) uint8_t ring[kPfStages][SB];
    __shared__ __attribute__((aligned(16))) uint8_t bfs[F8 ? 2 : 1][F8 ? kPfStageBytes : 16];
    const AttnArgs &a = pa.a;
    const PoolGeom &g = a.g;
    // one workgroup per (sequence, row pass, kv head): a long chunk's passes
    // run in parallel, each over the keys its own rows can see
    const int item = blockIdx.x / g.hkv;
    const int kvh = blockIdx.x % g.hkv;
    // the pass's record: one scalar load before the union and the first copies
    const int32_t *rec = pa.items + (int64_t)item * kPfItem;
    const int pass = scalar_ld(rec, 0);
    const int tok0 = scalar_ld(rec, 1);
    const int ntok = scalar_ld(rec, 2);
    const int sid = scalar_ld(rec, 3);
    const int pos0 = scalar_ld(rec, 4);
    const int row_t0 = scalar_ld(rec, 5);  // io rows of the sequence: row_t0 + j
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ln16 = lane & 15, lg = lane >> 4;
    const int n_rows = ntok * G;
    const int pass_row0 = pass * pa.pass_rows;
    const int pass_end = min(n_rows, pass_row0 + pa.pass_rows);  // rows [pass_row0, pass_end)
    // query positions spanned by this pass's rows
    const int tq_min = pos0 + pass_row0 / G;
    const int tq_max = pos0 + (pass_end - 1) / G;
    const int32_t *trow = g.table + (int64_t)sid * g.row_len;
    const uint8_t *layer_base = g.kv + (int64_t)a.layer * g.layer_stride + (int64_t)kvh * g.head_stride;
    const uint64_t lb_u = uniform64((uint64_t)(uintptr_t)layer_base);
    const uint64_t zp_u = uniform64((uint64_t)(uintptr_t)pa.zero_page);
    const uint32_t ring0 = lds_addr(&ring[0][0]);

    // union of the visible sets of the pass's queries: sinks, then the ring
    // run [A, tq_max] with A = max(S, tq_min - W + 1) (empty while every
    // query position is still below S)
    const int sink_tokens = min(g.n_sink, tq_max + 1);
    const int n_sb = (sink_tokens + kBlock - 1) / kBlock;
    const int A = g.window < 0 ? 0 : max(g.n_sink, tq_min - g.window + 1);
    const int ring_n = max(0, tq_max - A + 1);
    const int first = g.window < 0 ? A : (A - g.n_sink) % g.ring;
    const int first_off = first % kBlock;
    const int rb_start = first / kBlock;
    const int ring_blocks = g.ring / kBlock;
    const int n_rb = ring_n > 0 ? (first_off + ring_n + kBlock - 1) / kBlock : 0;
    const int last_hi = ring_n > 0 ? (first_off + ring_n - 1) % kBlock + 1 : kBlock;
    const int ring_p0 = A - first_off;
    const int nvb = n_sb + n_rb;
    const int n_stages = (nvb + 1) / 2;

    auto vblock = [&](int v) {
        PfBlock m;
        if (v < n_sb) {
            m.lb = v;
            m.lo = 0;
            m.hi = min(kBlock, sink_tokens - v * kBlock);
            m.p0 = v * kBlock;
            m.sink = true;
        } else if (v < nvb) {
            const int u = v - n_sb;
            int rb = rb_start + u;
            rb = rb >= ring_blocks ? rb - ring_blocks : rb;
            m.lb = g.n_sink_blocks + rb;
            m.lo = u == 0 ? first_off : 0;
            m.hi = u == n_rb - 1 ? last_hi : kBlock;
            m.p0 = ring_p0 + u * kBlock;
            m.sink = false;
        } else {
            m.lb = -1;
            m.lo = m.hi = m.p0 = 0;
            m.sink = false;
        }
        return m;
    };

    // The DMA of every stage is issued by DW waves: DMA wave i moves part of
    // block i & 1, the other waves only meet them at the barrier.  Lane
    // source offsets inside the block and the LDS offsets of the
    // instructions inside a ring slot are the same for every stage.  A block
    // takes NDI instructions -- bf16: 4 for the K tile, 4 for the V^T tile;
    // F8: 4 for the K and V codes, one 2-lane instruction for the 32 exponent
    // bytes -- and DMA wave i issues those k = (i >> 1) + (DW / 2) m, m < NPW.
    constexpr int NDI = F8 ? 5 : 8;  // DMA instructions per block
    constexpr int DW = F8 ? 2 : MTN_PF_DMA_WAVES;
    constexpr int NPW = NDI / (DW / 2);  // DMA instructions per DMA wave per stage
    static_assert(DW >= 2 && NPW * (DW / 2) == NDI, "DMA split");
    // The DMA waves are waves 2 and 3: with waves w and w + 4 sharing a SIMD,
    // at 200 rows per pass their SIMDs carry a one-tile second wave, while the
    // SIMD of waves 0 and 4 holds four tiles (measured 2.6 % per layer against
    // waves 0 and 1).
    constexpr int kDma0 = 2;
    static_assert(kPfWaves % 2 == 0 && kDma0 + DW <= kPfWaves / 2,
                  "DMA waves in the first half of the workgroup");
    const bool dma_wave = wv >= kDma0 && wv < kDma0 + DW;
    const int dwi = dma_wave ? wv - kDma0 : 0;
    const int db = dwi & 1;
    uint32_t dsrc[NPW], ddst[NPW];
#pragma unroll
    for (int m = 0; m < NPW; ++m) {
        const int j = (dwi >> 1) + (DW / 2) * m;
        if constexpr (F8) {
            dsrc[m] = j < 4 ? j * 1024 + lane * 16 : kF8Exp + (lane & 1) * 16;
            ddst[m] = db * kF8Read + (j < 4 ? j * 1024 : kF8Exp);
        } else {
            const int off = j < 4 ? db * 4096 + j * 1024 : 8192 + db * 4096 + (j - 4) * 1024;
            int bb;
            dsrc[m] = stage_src(off + lane * 16, &bb);
            ddst[m] = off;
        }
    }
    // logical block of virtual block v < nvb (branch-free: sinks, then the ring)
    auto vlb = [&](int v) {
        int rb = rb_start + v - n_sb;
        rb = rb >= ring_blocks ? rb - ring_blocks : rb;
        return v < n_sb ? v : g.n_sink_blocks + rb;
    };
    // physical block of virtual block v; -1 past the key union.  Every block
    // of the union holds appended tokens, so the planner has assigned it.
    auto phys = [&](int v) { return v < nvb ? scalar_ld(trow, vlb(v)) : -1; };
    // this wave's block of stage st into the stage's ring slot; stages past
    // the last (and absent blocks) move the zero page, so every stage costs
    // a DMA wave the same NPW instructions and its waits are constant
    auto issue_block = [&](int st, int ph) {
        // the block's address is formed in SGPRs: a vector copy of it was
        // spilled with one query head per kv head (fp8), and a spill reload
        // here waits for every DMA in flight
        const uint64_t src_u = ph >= 0 ? lb_u + (uint64_t)((int64_t)ph * g.block_stride) : zp_u;
        const uint8_t *src = (const uint8_t *)(uintptr_t)src_u;
        const uint32_t dst = ring0 + (uint32_t)((st % kPfStages) * SB);
#pragma unroll
        for (int m = 0; m < NPW; ++m) {
            if (F8 && m == 4) {
                // the lane offset is recomputed here rather than kept: with
                // one query head per kv head the fp8 kernel otherwise spills
                // it, and the reload's wait also drains the DMA ring
                if (lane < 2) dma16_s(kF8Exp + (lane & 1) * 16, src, dst + ddst[m]);
            } else {
                dma16_s(dsrc[m], src, dst + ddst[m]);
            }
        }
    };

    // per-lane LDS offsets inside a stage: K rows of the two QK MFMAs
    // (permuted keys), and the lane's V^T chunk
    // (the two MFMAs' keys differ by 4, which kswz ignores: MFMA 1's row is
    // MFMA 0's plus 4 * 256 bytes)
    int koff[4];
    {
        const int kap = 8 * (ln16 >> 2) + (ln16 & 3);
#pragma unroll
        for (int s = 0; s < 4; ++s) koff[s] = lds_k(kap >> 4, kap & 15, s * 4 + lg);
    }
    const int lblk = lg >> 1;          // the block of this lane's eight keys
    const int lkey0 = 8 * (lg & 1);    // ... and the first of them
    const int voff = lds_v16(lblk, ln16, lg & 1);  // + dt * 16 * 32 for d tile dt

    const int hq0 = kvh * G;
    // Fused chunk append (fp8 pool; a.k_new set).  The host passes it only
    // when every sequence of the plan takes one row pass, so no other
    // workgroup reads this sequence's blocks of this kv head.  (For the bf16
    // pool the separate append launch measured as fast, so that kernel has no
    // such path.)  The waves that issue no copies rotate K, quantize K and V
    // and store the sequence's tokens: their first batch of loads goes out
    // just ahead of the query loads, the stores follow the query rotation.
    // When the chunk's first token lies in a stage that the prologue copies
    // (a short sequence), or that is copied at the first two stage barriers,
    // those copies wait behind the completed stores and a barrier.  Otherwise
    // that copy is issued at a later stage barrier, and the stores, issued
    // before the first one by waves of this workgroup, are ordered before it
    // at workgroup scope.  A copy of the ring block that also holds the
    // window's oldest keys may meet the append's stores to its other slots:
    // those slots are masked there.
    const bool fuse = F8 && a.k_new != nullptr;
    bool early_chunk = false;
    if (fuse) {
        const int cv = pos0 < sink_tokens ? pos0 / kBlock : n_sb + (pos0 - ring_p0) / kBlock;
        early_chunk = cv / 2 < kPfStages + 1;  // copied by the prologue or at barrier 0 or 1
    }
    constexpr int NAW = kPfWaves - DW;          // appending waves
    constexpr int AB = 4;                       // tokens per batch (more spill across the loops)
    const int aw = wv < kDma0 ? wv : wv - DW;   // this wave's index among them
    // The loads keep the raw bf16 bits: converted on load, the compiler
    // consumed each value right away and waited for every load in turn
    // (four memory round trips before the query loads went out).
    struct AppBatch {
        uint32_t k0[AB], k1[AB], v0[AB], v1[AB];  // bf16 bits, zero-extended
        float2 cs[AB];
        int blk[AB], off[AB];
    };
    // tokens j0, j0 + NAW, ... (indices clamped into the sequence)
    auto app_load = [&](int j0, AppBatch &b) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < AB; ++u) {
            const int j = min(j0 + u * NAW, ntok - 1);
            const int t = tok0 + j;
            const int64_t ri = ((int64_t)(row_t0 + j) * g.hkv + kvh) * D;
            const uint16_t *kr = (const uint16_t *)a.k_new + ri;
            const uint16_t *vr = (const uint16_t *)a.v_new + ri;
            b.k0[u] = kr[lane];
            b.k1[u] = kr[lane + 64];
            b.v0[u] = vr[lane];
            b.v1[u] = vr[lane + 64];
            b.cs[u] = a.p.rope[(int64_t)t * (D / 2) + lane];
            b.blk[u] = scalar_ld(a.p.tok_block, t);
            b.off[u] = scalar_ld(a.p.tok_off, t);
        }
    };
    auto app_store = [&](int j0, AppBatch &b) __attribute__((always_inline)) {
        uint8_t *lw = const_cast<uint8_t *>(layer_base);
        auto f = [](uint32_t bits) { return __uint_as_float(bits << 16); };
        // every use of the loaded values stays here: without the pins the
        // compiler moved their conversions up beside the loads
#pragma unroll
        for (int u = 0; u < AB; ++u)
            asm volatile("" : "+v"(b.k0[u]), "+v"(b.k1[u]), "+v"(b.v0[u]), "+v"(b.v1[u]));
#pragma unroll
        for (int u = 0; u < AB; ++u) {
            if (j0 + u * NAW >= ntok) break;
            const float k0 = f(b.k0[u]), k1 = f(b.k1[u]);
            const float y0 = fmaf(k0, b.cs[u].x, -k1 * b.cs[u].y);
            const float y1 = fmaf(k1, b.cs[u].x, k0 * b.cs[u].y);
            store_token_fp8(lw + (int64_t)b.blk[u] * g.block_stride, b.off[u], y0, y1,
                            f(b.v0[u]), f(b.v1[u]), lane);
        }
    };
    {
        // ring blocks every row of the pass sees whole: [fr_lo, fr_hi) (as
        // virtual indices)
        int fr_lo, fr_hi;
        {
            // ring block u spans positions ring_p0 + 16u .. + 15; it is whole
            // when u > 0 or first_off == 0, u < n_rb - 1 or last_hi == 16,
            // its end is at most tq_min and (windowed) its start is at least
            // tq_max - W + 1
            int ulo = first_off == 0 ? 0 : 1;
            if (g.window >= 0) {
                const int need = tq_max - g.window + 1 - ring_p0;  // p0 offset >= need
                ulo = max(ulo, need <= 0 ? 0 : (need + kBlock - 1) / kBlock);
            }
            const int lim = tq_min - (kBlock - 1) - ring_p0;      // 16u <= lim
            int uhi = lim < 0 ? 0 : lim / kBlock + 1;
            uhi = min(uhi, last_hi == kBlock ? n_rb : n_rb - 1);
            fr_lo = n_sb + ulo;
            fr_hi = n_sb + max(uhi, ulo);
        }
        // ---- per-wave query tiles: rows r = pass_row0 + (wv + kPfWaves i) * 16 + ln16
        uint4 qf[kPfTpw][4];
        f32x4_t acc[kPfTpw][8];
        // row reference max (log2 units) and the row sum of the probabilities.
        // bf16 pool: the sum of their bf16 roundings, accumulated by an MFMA
        // against all-ones (every entry = the row sum).  fp8 pool: ls holds
        // the lane's part of the fp32 sum (its eight keys of every
        // stage), the four lanes of a row added in the epilogue; vector adds
        // in place of that MFMA free registers the fp8 stage loop otherwise
        // spills (2-3 % per layer; the bf16 kernel measured no gain).  The reference starts at the lowest finite float: the first finite
        // score of a row exceeds it by more than 2^8 and sets it, while
        // masked (-inf) scores give probability 0 against it.
        float m_ref[kPfTpw];
        // bf16 pool: the QK MFMAs start their accumulators at -msh, so the
        // scores come out already shifted by the reference and each
        // probability is one exponential with no subtraction; thr is the bump
        // threshold on shifted scores (m_ref - msh + 2^8: 2^8 once the first
        // finite score has set the reference).  The fp8 kernel keeps unshifted
        // scores (msh stays 0, thr = m_ref + 2^8): its conversion stage leaves
        // no registers for the four shift values per tile (measured 0.386 ->
        // 0.495 ms per layer with them, from spills inside the stage loops).
        constexpr bool kShift = !F8;
        float msh[kPfTpw], thr[kPfTpw];
        f32x4_t csh[kPfTpw];  // {-msh} x 4, kept so the QK start needs no moves
        constexpr bool kMfmaSum = !F8;
        f32x4_t l_i[kPfTpw];
        float ls[kPfTpw];
        int tq_i[kPfTpw];
        bool live[kPfTpw];
        // The tiles' loads go out together, ahead of any rotation: every q dim
        // pair and (cos, sin) pair of both tiles (the io rows follow from the
        // pass record), then the arithmetic.  (Interleaved with the rotation,
        // with the io row loaded first, the loads took one memory round trip
        // per slice: about 10 us of every workgroup's prologue.)  Slices s and
        // s + 2 share their (cos, sin) pairs (dims d and d + 64 hold one
        // rotation pair).
        int tq_j[kPfTpw], gh_i[kPfTpw];
        bool rv_i[kPfTpw];
        int64_t row_i[kPfTpw];
#pragma unroll
        for (int i = 0; i < kPfTpw; ++i) {
            const int tile0 = pass_row0 + (wv + kPfWaves * i) * 16;
            live[i] = tile0 < pass_end;
            const int r = tile0 + ln16;
            rv_i[i] = r < pass_end;
            tq_j[i] = rv_i[i] ? r / G : 0;
            gh_i[i] = rv_i[i] ? r % G : 0;
            tq_i[i] = pos0 + tq_j[i];
            row_i[i] = row_t0 + tq_j[i];  // no load before the q loads
            m_ref[i] = -3.402823466e38f;
            msh[i] = 0.f;
            csh[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            thr[i] = m_ref[i] + 8.f;
            l_i[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            ls[i] = 0.f;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) acc[i][dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
        uint4 qx[kPfTpw][4], qy[kPfTpw][4];  // dims d0 .. d0 + 7 and their partners d0 ^ 64
        float4 qc[kPfTpw][2][4];             // (cos, sin) of dims (d0 & 63) .. + 7
        AppBatch ab;
        if (fuse && !dma_wave) app_load(aw, ab);
        __builtin_amdgcn_sched_barrier(0);  // the query loads follow at once
#pragma unroll
        for (int i = 0; i < kPfTpw; ++i) {
            const int t = tok0 + tq_j[i];
            const bf16_t *qh = (const bf16_t *)a.q + (row_i[i] * g.hq + hq0 + gh_i[i]) * D;
            const float2 *rp = a.p.rope + (int64_t)t * (D / 2);
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int d0 = s * 32 + 8 * lg;
                qx[i][s] = *(const uint4 *)(qh + d0);
                qy[i][s] = *(const uint4 *)(qh + (d0 ^ 64));
            }
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
                for (int k = 0; k < 4; ++k) qc[i][h2][k] = ((const float4 *)(rp + h2 * 32 + 8 * lg))[k];
        }
        // The DMA waves copy the first kPfEarly stages right behind the q
        // loads: the first barriers need them, and the rotation's waits for
        // the q loads (counted by the compiler, which does not see the copies)
        // then cover exactly these copies.  The rest of the ring follows the
        // rotation.
        if (dma_wave && !early_chunk) {
#pragma unroll
            for (int st = 0; st < kPfEarly; ++st) issue_block(st, phys(2 * st + db));
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < kPfTpw; ++i) {
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                // dims d0 + e, e < 8, d0 = s*32 + 8*lg; RoPE partner is d +- 64
                const int d0 = s * 32 + 8 * lg;
                float xv[8], yv[8], cs[16];
                unpack8(qx[i][s], xv);
                unpack8(qy[i][s], yv);
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const float4 c = qc[i][s & 1][k];
                    cs[4 * k] = c.x;
                    cs[4 * k + 1] = c.y;
                    cs[4 * k + 2] = c.z;
                    cs[4 * k + 3] = c.w;
                }
                const float sg = d0 < 64 ? -1.f : 1.f;
                // rows past the pass become zero queries; a mask rather than a
                // select, so that the compiler keeps the loads unconditional
                const uint32_t keep = rv_i[i] ? 0xFFFFFFFFu : 0u;
                uint32_t w[4];
#pragma unroll
                for (int e = 0; e < 8; e += 2) {
                    float r2[2];
#pragma unroll
                    for (int u = 0; u < 2; ++u)
                        r2[u] = fmaf(xv[e + u], cs[2 * (e + u)], sg * yv[e + u] * cs[2 * (e + u) + 1]) *
                                a.scale_log2;
                    w[e / 2] = pack_bf16x2(r2[0], r2[1]) & keep;
                }
                // computed here, before the DMA waves issue the ring: the
                // compiler's waits for these loads count only its own loads, so
                // left after the copies they would wait for most of the ring
#pragma unroll
                for (int e = 0; e < 4; ++e) asm volatile("" : "+v"(w[e]));
                qf[i][s] = make_uint4(w[0], w[1], w[2], w[3]);
            }
        }

        // The stage loop is software-pipelined by one stage: iteration st
        // masks and softmaxes the scores of stage st (computed by the previous
        // iteration) while the QK MFMAs of stage st + 1 run, then accumulates
        // PV of stage st.  The softmax keeps a per-row reference max that
        // moves only when a score exceeds it by more than 2^8 (probabilities
        // stay <= 256), so the accumulator rescale is rare; the result is the
        // same softmax.  Whether any lane holds such a score is checked on
        // the lane's own eight scores; only then is the row max formed across
        // the four lanes of a row.
        constexpr float kLazy = 8.f;
        // the bf16 stage buffer the MFMAs read for stage st
        auto stage_buf = [&](int st) -> uint8_t * {
            if constexpr (F8)
                return &bfs[st & 1][0];
            else
                return &ring[st % kPfStages][0];
        };
        // FULL stages: both blocks in the key union and inside the ring blocks
        // every row sees whole
        const int full_r_lo = (fr_lo + 1) / 2, full_r_hi = min(fr_hi, nvb) / 2;
        // V^T words of slots outside a block's valid range (they may hold
        // NaN, and 0 * NaN is NaN) are zeroed in registers: the lane's V
        // chunk holds slots lkey0 .. lkey0 + 7 of block lblk for one d, two
        // per dword (the even slot in the low half)
        auto v_slot_mask = [&](int st, uint32_t (&vm)[4]) {
            const PfBlock mb = vblock(2 * st + lblk);
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int ka = lkey0 + 2 * q4, kb = ka + 1;
                vm[q4] = ((ka >= mb.lo && ka < mb.hi) ? 0x0000FFFFu : 0u) |
                         ((kb >= mb.lo && kb < mb.hi) ? 0xFFFF0000u : 0u);
            }
        };
        // lane l holds row ln16 and stage keys 8 lg + r (sa) and 8 lg + 4 + r
        // (sb), r < 4: slots lkey0 + r and lkey0 + 4 + r of block lblk.
        // Scores of slots the row's query cannot see become -inf.
        auto mask_scores = [&](auto nt_c, int st, f32x4_t (&sa)[kPfTpw], f32x4_t (&sb)[kPfTpw])
                               __attribute__((always_inline)) {
            constexpr int NT = decltype(nt_c)::value;
            const PfBlock mb = vblock(2 * st + lblk);
            const int bp0 = mb.p0, blo = mb.lo, bhi = mb.hi;
#pragma unroll
            for (int i = 0; i < NT; ++i) {
                // visible slots of the block for query position tq: one range
                const int tq = tq_i[i];
                const int wl = g.window < 0 ? -(1 << 30) : tq - g.window + 1;
                const int vlo = mb.sink ? blo : max(blo, wl - bp0);
                const int vhi = min(bhi, tq + 1 - bp0);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int oa = lkey0 + r, ob = oa + 4;
                    sa[i][r] = (oa >= vlo && oa < vhi) ? sa[i][r] : -INFINITY;
                    sb[i][r] = (ob >= vlo && ob < vhi) ? sb[i][r] : -INFINITY;
                }
            }
        };
        // S^T of a stage for every tile of this wave (K fragments read once,
        // shared by the tiles; tiles past the last row compute on zero
        // queries and are dropped)
        auto qk = [&](auto nt_c, const uint8_t *sm, f32x4_t (&sa)[kPfTpw], f32x4_t (&sb)[kPfTpw])
                      __attribute__((always_inline)) {
            constexpr int NT = decltype(nt_c)::value;
#pragma unroll
            for (int i = 0; i < NT; ++i) {
                sa[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
                sb[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const uint4 k0 = *(const uint4 *)(sm + koff[s]);
                const uint4 k1 = *(const uint4 *)(sm + koff[s] + 1024);
#pragma unroll
                for (int i = 0; i < NT; ++i) {
                    sa[i] = mfma16x16x32(k0, qf[i][s], sa[i]);
                    sb[i] = mfma16x16x32(k1, qf[i][s], sb[i]);
                }
            }
        };
        if (fuse) {
            if (!dma_wave) {
                app_store(aw, ab);
                for (int j0 = aw + AB * NAW; j0 < ntok; j0 += AB * NAW) {
                    app_load(j0, ab);
                    app_store(j0, ab);
                }
                // copies issued right after the next barrier read them: the
                // stores are acknowledged by the L2 first
                if (early_chunk) vm_wait<0>();
            }
            if (early_chunk) {
                __syncthreads();
                if (dma_wave) {
#pragma unroll
                    for (int st = 0; st < kPfEarly; ++st) issue_block(st, phys(2 * st + db));
                }
            }
        }
        // ring prologue: stages kPfEarly .. kPfStages - 2 join the first ones in flight
        int nph = -1;  // DMA waves: physical block of the next stage to issue
        if (dma_wave) {
#pragma unroll
            for (int st = kPfEarly; st < kPfStages - 1; ++st) issue_block(st, phys(2 * st + db));
            nph = phys(2 * (kPfStages - 1) + db);
        }
        f32x4_t sa[kPfTpw], sb[kPfTpw];  // scores of the stage being consumed
        // Ping-pong (bf16): the second half of the waves (group B) meets the
        // stage barrier after its QK MFMAs and exponentials instead of before
        // them, so it runs half a stage ahead of group A: while one wave of a
        // SIMD streams PV MFMAs, the other runs its LDS reads, maximum test and
        // exponentials (measured 4-5 % per layer).  Group B then reads the K
        // tiles of stage st + 1 before barrier st, so the DMA waves (all in
        // group A) wait one stage further ahead: stages 0 and 1 here, st + 2
        // at barrier st.  The ring slot refilled after barrier st held stage
        // st - 1, which both groups finished before reaching it.  The fp8
        // kernel keeps the common barrier: its conversion step is a second
        // workgroup-wide exchange per stage.
        constexpr bool kPP = !F8;
        const bool grp_b = kPP && wv >= kPfWaves / 2;
        if (dma_wave) vm_wait<NPW * (kPfStages - (kPP ? 3 : 2))>();  // stage 0 (and 1) landed
        __syncthreads();
        if constexpr (F8) {
            f8_stage_to_bf16(&ring[0][0], stage_buf(0), tid);
            __syncthreads();
        }
        // one stage; MASKED: the stage may hold keys some row cannot see
        auto step = [&](auto nt_c, int st, auto masked_c) __attribute__((always_inline)) {
            constexpr int NT = decltype(nt_c)::value;
            constexpr bool MASKED = decltype(masked_c)::value;
            const uint8_t *sm = stage_buf(st);
            // V^T chunks of stage st (visible since the previous barrier):
            // their LDS latency overlaps the wait below
            uint4 vf[8];
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) vf[dt] = *(const uint4 *)(sm + voff + dt * 16 * 32);
            if constexpr (MASKED) {
                mask_scores(nt_c, st, sa, sb);
                uint32_t vm[4];
                v_slot_mask(st, vm);
#pragma unroll
                for (int dt = 0; dt < 8; ++dt)
                    vf[dt] = make_uint4(vf[dt].x & vm[0], vf[dt].y & vm[1], vf[dt].z & vm[2], vf[dt].w & vm[3]);
            }
            // stage st + 1 (ping-pong: st + 2) landed (zero-page stages after
            // the last); the barrier covers both DMA waves and frees the ring
            // slot last read at st - 1, which takes stage st + kPfStages - 1
            if (!grp_b) {
                if (dma_wave) vm_wait<NPW * (kPfStages - (kPP ? 4 : 3))>();
                __syncthreads();
                if (dma_wave) {
                    const int nst = st + kPfStages - 1;
                    issue_block(nst, nph);
                    nph = phys(2 * (nst + 1) + db);
                }
            }
            if constexpr (F8) {
                // the other bf16 buffer: its stage (st - 1) is consumed
                f8_stage_to_bf16(&ring[(st + 1) % kPfStages][0], stage_buf(st + 1), tid);
                __syncthreads();
            }
            // K fragments of stage st + 1.  bf16: read before the max test, whose
            // instructions then cover their LDS latency (2.7-7.5 % per layer);
            // fp8 measured no gain, its reads stay with the QK MFMAs
            const uint8_t *nsm = stage_buf(st + 1);
            uint4 kf[4][2];
            auto load_kf = [&]() __attribute__((always_inline)) {
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    kf[s][0] = *(const uint4 *)(nsm + koff[s]);
                    kf[s][1] = *(const uint4 *)(nsm + koff[s] + 1024);
                }
            };
            if constexpr (!F8) load_kf();
            // lazy reference max: lane-local test, row max only on a bump
            float m8[kPfTpw];
            bool bump = false;
#pragma unroll
            for (int i = 0; i < NT; ++i) {
                // three-operand maxima only (a two-operand one costs the
                // compiler two NaN-quieting instructions); sa[i][0] twice
                m8[i] = vmax3(vmax3(sa[i][0], sa[i][1], sa[i][2]), vmax3(sa[i][3], sb[i][0], sb[i][1]),
                              vmax3(sb[i][2], sb[i][3], sa[i][0]));
                bump = bump || m8[i] > thr[i];
            }
            if (__builtin_amdgcn_ballot_w64(bump)) {
#pragma unroll
                for (int i = 0; i < NT; ++i) {
                    // true row max of the stage, the new reference, and the
                    // re-shift of this stage's (already shifted) scores
                    const float mx = rows_max(m8[i]) + msh[i];
                    const bool up = mx > m_ref[i] + kLazy;
                    const float mnew = up ? mx : m_ref[i];
                    const float alpha = up ? __builtin_amdgcn_exp2f(m_ref[i] - mnew) : 1.f;
                    m_ref[i] = mnew;
                    if constexpr (kShift) {
                        const float dsh = up ? mnew - msh[i] : 0.f;
                        msh[i] = up ? mnew : msh[i];
                        csh[i] = f32x4_t{-msh[i], -msh[i], -msh[i], -msh[i]};
                        thr[i] = up ? kLazy : thr[i];
                        sa[i] -= dsh;
                        sb[i] -= dsh;
                    } else {
                        thr[i] = mnew + kLazy;
                    }
                    if constexpr (kMfmaSum)
                        l_i[i] *= alpha;  // all four entries
                    else
                        ls[i] *= alpha;
#pragma unroll
                    for (int dt = 0; dt < 8; ++dt) acc[i][dt] *= alpha;
                }
            }
            // QK of the next stage (at the last stage it reads a stale
            // buffer and its scores are dropped), interleaved with this
            // stage's probabilities: in each of four groups, one MFMA then
            // two VALU instructions, so the exponentials run while the matrix
            // core works
            if constexpr (F8) load_kf();
            f32x4_t na[kPfTpw], nb[kPfTpw];
            float p[kPfTpw][8];
            constexpr int kEpg = 2 * NT;  // probabilities per group
#pragma unroll
            for (int s = 0; s < 4; ++s) {
#pragma unroll
                for (int i = 0; i < NT; ++i) {
                    const f32x4_t c0 = kShift ? csh[i] : f32x4_t{0.f, 0.f, 0.f, 0.f};
                    na[i] = mfma16x16x32(kf[s][0], qf[i][s], s ? na[i] : c0);
                    nb[i] = mfma16x16x32(kf[s][1], qf[i][s], s ? nb[i] : c0);
                }
#pragma unroll
                for (int u = 0; u < kEpg; ++u) {
                    const int f = s * kEpg + u, i = f >> 3, e = f & 7;
                    const float sc = e < 4 ? sa[i][e] : sb[i][e - 4];
                    p[i][e] = __builtin_amdgcn_exp2f(kShift ? sc : sc - m_ref[i]);
                    // keep it in this group: without the pin the compiler sinks every
                    // exponential below the last group, after the QK MFMAs
                    asm volatile("" : "+v"(p[i][e]));
                }
#ifndef MTN_PF_NO_SCHED
                if (s == 0) __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);  // all K reads first
#pragma unroll
                for (int k = 0; k < 2 * NT; ++k) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x402, 2, 0);  // VALU or TRANS
                }
                __builtin_amdgcn_sched_barrier(0);
#endif
            }
            uint4 pb[kPfTpw];
#pragma unroll
            for (int i = 0; i < NT; ++i)
                pb[i] = make_uint4(pack_bf16x2(p[i][0], p[i][1]), pack_bf16x2(p[i][2], p[i][3]),
                                   pack_bf16x2(p[i][4], p[i][5]), pack_bf16x2(p[i][6], p[i][7]));
            if (grp_b) __syncthreads();  // group B's stage barrier
            // row sums: of the bf16 probabilities by an all-ones A operand, or
            // the lane's part by vector adds
            const uint4 ones = make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u);
#pragma unroll
            for (int i = 0; i < NT; ++i) {
                if constexpr (kMfmaSum)
                    l_i[i] = mfma16x16x32(ones, pb[i], l_i[i]);
                else
                    ls[i] += ((p[i][0] + p[i][1]) + (p[i][2] + p[i][3])) +
                             ((p[i][4] + p[i][5]) + (p[i][6] + p[i][7]));
            }
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) {
#pragma unroll
                for (int i = 0; i < NT; ++i) acc[i][dt] = mfma16x16x32(vf[dt], pb[i], acc[i][dt]);
            }
#pragma unroll
            for (int i = 0; i < NT; ++i) {
                sa[i] = na[i];
                sb[i] = nb[i];
            }
        };
        // the FULL stages inside the whole ring blocks run without masking;
        // every other stage (sinks, the window's left edge, the causal edge)
        // takes the masked step (exact for FULL stages too).  Three loops, so
        // each keeps its scores and accumulators in fixed registers.
        const int st_a = min(full_r_lo, n_stages);
        const int st_b = max(st_a, min(full_r_hi, n_stages));
        // NT: this wave's live tiles.  A wave whose second tile lies past the
        // pass's rows skips its MFMAs and exponentials; every wave still runs
        // the same barriers and DMA turns.
        auto run = [&](auto nt_c) __attribute__((always_inline)) {
            qk(nt_c, stage_buf(0), sa, sb);
            int st = 0;
            for (; st < st_a; ++st) step(nt_c, st, std::true_type{});
            for (; st < st_b; ++st) step(nt_c, st, std::false_type{});
            for (; st < n_stages; ++st) step(nt_c, st, std::true_type{});
        };
        if (kPfTpw == 1 || !live[kPfTpw - 1])
            run(std::integral_constant<int, 1>{});
        else
            run(std::integral_constant<int, kPfTpw>{});
        // no DMA may land in LDS after the workgroup has ended
        if (dma_wave) vm_wait<0>();

        // ---- epilogue: normalise and write rows of this pass
#pragma unroll
        for (int i = 0; i < kPfTpw; ++i) {
            if (!live[i]) continue;
            // (every lane of the wave takes part in the row sum)
            const float lt = kMfmaSum ? l_i[i][0] : rows_sum(ls[i]);
            const int r = pass_row0 + (wv + kPfWaves * i) * 16 + ln16;
            if (r >= pass_end) continue;
            const int j = r / G, gh = r % G;
            const int64_t row = row_t0 + j;
            bf16_t *ob = (bf16_t *)a.out + (row * g.hq + hq0 + gh) * D;
            const float inv = 1.f / lt;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) {
                const int d0 = dt * 16 + 4 * lg;
                uint2 w = make_uint2(pack_bf16x2(acc[i][dt][0] * inv, acc[i][dt][1] * inv),
                                     pack_bf16x2(acc[i][dt][2] * inv, acc[i][dt][3] * inv));
                *(uint2 *)(ob + d0) = w;
            }
            if (a.lse && lg == 0)
                a.lse[row * g.hq + hq0 + gh] =
                    (m_ref[i] + __builtin_amdgcn_logf(lt)) * 0.6931471805599453f;
        }
    }
}

template <typename T, int D, int G>
hipError_t launch_valu_t(const AttnArgs &a, hipStream_t s) {
    using DS = DecodeShape<G>;
    int64_t units = (int64_t)a.p.n_tok * a.g.hkv * a.n_split;
    if (units == 0) return hipSuccess;
    if (units > INT32_MAX) return hipErrorInvalidValue;  // one grid dimension, 32-bit unit index
    hipLaunchKernelGGL((k_attn_valu<T, D, G, DS::WPU, DS::NG, DS::NBUF>), dim3((unsigned)units),
                       dim3(64 * DS::WPU * DS::NG), 0, s, a);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_valu_d(const AttnArgs &a, int G, hipStream_t s) {
    switch (G) {
        case 1: return launch_valu_t<T, D, 1>(a, s);
        case 2: return launch_valu_t<T, D, 2>(a, s);
        case 4: return launch_valu_t<T, D, 4>(a, s);
        case 8: return launch_valu_t<T, D, 8>(a, s);
        default: return hipErrorInvalidValue;
    }
}

template <typename T, int D, int G>
int resident_t() {
    using DS = DecodeShape<G>;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &n, k_attn_valu<T, D, G, DS::WPU, DS::NG, DS::NBUF>, 64 * DS::WPU * DS::NG, 0) !=
        hipSuccess)
        return 1;
    return n > 0 ? n : 1;
}
template <typename T, int D>
int resident_d(int G) {
    switch (G) {
        case 1: return resident_t<T, D, 1>();
        case 2: return resident_t<T, D, 2>();
        case 4: return resident_t<T, D, 4>();
        default: return resident_t<T, D, 8>();
    }
}

}  // namespace

int attn_valu_resident_per_cu(int dtype, int d, int g) {
    if (!attn_valu_supported(dtype, d, g)) return 1;
    if (dtype == 1) return d == 128 ? resident_d<bf16_t, 128>(g) : resident_d<bf16_t, 64>(g);
    return d == 128 ? resident_d<float, 128>(g) : resident_d<float, 64>(g);
}

bool attn_valu_supported(int dtype, int d, int g) {
    if (g != 1 && g != 2 && g != 4 && g != 8) return false;
    if (d != 64 && d != 128) return false;
    return dtype == 0 || dtype == 1;
}

bool prefill_mfma_supported(int dtype, int d, int g) {
    return (dtype == 1 || dtype == 2) && d == 128 && (g == 1 || g == 2 || g == 4 || g == 8);
}

hipError_t launch_plan_apply(const int32_t *upd_idx, const int32_t *upd_val, int32_t n_upd,
                             int32_t *table, const int32_t *tok_pos, int32_t n_tok,
                             const double *inv_freq, int32_t half_d, float2 *rope,
                             hipStream_t s) {
    int64_t total = std::max<int64_t>((int64_t)n_tok * half_d, n_upd);
    if (total == 0) return hipSuccess;
    int64_t grid = std::min<int64_t>((total + 255) / 256, 4096);
    hipLaunchKernelGGL(k_plan_apply, dim3((unsigned)grid), dim3(256), 0, s, upd_idx, upd_val, n_upd,
                       table, tok_pos, n_tok, inv_freq, half_d, rope);
    return hipGetLastError();
}

hipError_t launch_append(int dtype, const PoolGeom &g, const PlanView &p, int32_t layer,
                         const void *k, const void *v, const int32_t *run_tok0,
                         const int32_t *run_len, int32_t n_runs, hipStream_t s) {
    if (g.d > 128) return hipErrorInvalidValue;  // the per-wave LDS tile holds D <= 128
    const int64_t groups = (int64_t)n_runs * g.hkv;
    if (groups == 0) return hipSuccess;
    if (groups > INT32_MAX) return hipErrorInvalidValue;
    const unsigned grid = (unsigned)groups;
    if (dtype == 1)
        hipLaunchKernelGGL(k_append<bf16_t>, dim3(grid), dim3(64 * kAppendWaves), 0, s, g, p, layer,
                           (const bf16_t *)k, (const bf16_t *)v, run_tok0, run_len);
    else
        hipLaunchKernelGGL(k_append<float>, dim3(grid), dim3(64 * kAppendWaves), 0, s, g, p, layer,
                           (const float *)k, (const float *)v, run_tok0, run_len);
    return hipGetLastError();
}

hipError_t launch_attn_valu(int dtype, const AttnArgs &a, hipStream_t s) {
    const int G = a.g.hq / a.g.hkv;
    if (!attn_valu_supported(dtype, a.g.d, G)) return hipErrorInvalidValue;
    if (dtype == 1) {
        return a.g.d == 128 ? launch_valu_d<bf16_t, 128>(a, G, s) : launch_valu_d<bf16_t, 64>(a, G, s);
    }
    return a.g.d == 128 ? launch_valu_d<float, 128>(a, G, s) : launch_valu_d<float, 64>(a, G, s);
}

hipError_t launch_merge(int dtype, const AttnArgs &a, hipStream_t s) {
    int64_t n = (int64_t)a.p.n_tok * a.g.hq;
    if (n == 0) return hipSuccess;
    if (dtype == 1) {
        if (a.g.d == 128)
            hipLaunchKernelGGL((k_merge<bf16_t, 128>), dim3((unsigned)n), dim3(64), 0, s, a);
        else
            hipLaunchKernelGGL((k_merge<bf16_t, 64>), dim3((unsigned)n), dim3(64), 0, s, a);
    } else {
        if (a.g.d == 128)
            hipLaunchKernelGGL((k_merge<float, 128>), dim3((unsigned)n), dim3(64), 0, s, a);
        else
            hipLaunchKernelGGL((k_merge<float, 64>), dim3((unsigned)n), dim3(64), 0, s, a);
    }
    return hipGetLastError();
}

// Device address of `scratch` on the current device, resolved once per device
// (the array's host-side name is not a device address).
hipError_t scratch_buffer(float **ptr, size_t *floats) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static float *addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = (float *)p;
    }
    *ptr = addr[dev];
    *floats = kScratchFloats;
    return hipSuccess;
}

int prefill_rows_per_pass() { return kPfRowsPerPass; }
// a pass covers a whole number of wave tiles of every wave: 128 rows (one
// tile per wave) or the full kPfRowsPerPass
bool prefill_pass_rows_valid(int rows) { return rows == kPfRowsPerPass || rows == kPfWaves * 16; }

template <bool F8>
void launch_prefill_g(int G, dim3 grid, dim3 block, hipStream_t s, const PfArgs &pa) {
    switch (G) {
        case 1: hipLaunchKernelGGL((k_prefill_mfma<1, F8>), grid, block, 0, s, pa); break;
        case 2: hipLaunchKernelGGL((k_prefill_mfma<2, F8>), grid, block, 0, s, pa); break;
        case 4: hipLaunchKernelGGL((k_prefill_mfma<4, F8>), grid, block, 0, s, pa); break;
        default: hipLaunchKernelGGL((k_prefill_mfma<8, F8>), grid, block, 0, s, pa); break;
    }
}

hipError_t launch_prefill_mfma(int dtype, const AttnArgs &a, const int32_t *items, int32_t n_items,
                               int32_t pass_rows, const uint8_t *zero_page, hipStream_t s) {
    const int G = a.g.hq / a.g.hkv;
    if (!prefill_mfma_supported(dtype, a.g.d, G) || n_items <= 0 || !zero_page || !items ||
        !prefill_pass_rows_valid(pass_rows))
        return hipErrorInvalidValue;
    if (((uintptr_t)items & 31) != 0) return hipErrorInvalidValue;  // records are 32-byte aligned
    if ((a.k_new == nullptr) != (a.v_new == nullptr) || (a.k_new && dtype != 2))
        return hipErrorInvalidValue;  // the fused append is the fp8 kernel's
    PfArgs pa{a, items, zero_page, pass_rows};
    dim3 grid((unsigned)(n_items * a.g.hkv)), block(64 * kPfWaves);
    if (dtype == 2)
        launch_prefill_g<true>(G, grid, block, s, pa);
    else
        launch_prefill_g<false>(G, grid, block, s, pa);
    return hipGetLastError();
}

hipError_t launch_poison(int dtype, const PoolGeom &g, int32_t n_layers, int64_t n_blocks,
                         const uint16_t *live, hipStream_t s) {
    unsigned grid = 8192;
    if (dtype == 1)
        hipLaunchKernelGGL(k_poison<bf16_t>, dim3(grid), dim3(256), 0, s, g, n_layers, n_blocks, live);
    else
        hipLaunchKernelGGL(k_poison<float>, dim3(grid), dim3(256), 0, s, g, n_layers, n_blocks, live);
    return hipGetLastError();
}

hipError_t launch_copy(const void *src, void *dst, size_t bytes, hipStream_t s) {
    int64_t n = (int64_t)(bytes / 16);
    if (n == 0) return hipSuccess;
    int64_t grid = std::min<int64_t>((n + 255) / 256, 256 * 16);
    hipLaunchKernelGGL(k_copy, dim3((unsigned)grid), dim3(256), 0, s, (const u32x4_t *)src,
                       (u32x4_t *)dst, n);
    return hipGetLastError();
}

hipError_t launch_read(const void *src, size_t bytes, uint32_t *out, hipStream_t s) {
    const int64_t n = (int64_t)(bytes / 8192);  // whole 8 KiB chunks
    if (n == 0) return hipSuccess;
    int dev = 0, n_cu = 256;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
    const int64_t grid = std::min<int64_t>((n + kReadWaves - 1) / kReadWaves, 2 * (int64_t)n_cu);
    hipLaunchKernelGGL(k_read, dim3((unsigned)grid), dim3(64 * kReadWaves), 0, s,
                       (const uint8_t *)src, n, out);
    return hipGetLastError();
}

}  // namespace mtn
