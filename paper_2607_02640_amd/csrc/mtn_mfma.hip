// gfx950 MFMA decode attention over KV blocks in bf16 or in FP8 (E4M3 codes
// with one power-of-two scale per (token, kv head) and tensor), with the
// append fusable, plus the FP8 pool's fused RoPE + quantize + append and its
// debug poison.
//
// Method: Metronome (arXiv 2607.02640) §4.1 / App. A for what a query sees
// (sinks ∪ the W positions ending at it, causal).  Per-token KV reduction
// composes with that bound (§4.1, closing remark; §6): the window bounds how
// many tokens stay resident, the 8-bit codes how many bytes each one holds.
//
// FP8 layout of one (layer, block, kv head) region, D = 128, head stride 4224:
//   [0, 2048)     K codes, [16 keys][128 dims]
//   [2048, 4096)  V codes in key quads: byte ((key / 4) * 128 + d) * 4 + key % 4
//   [4096, 4112)  K scale exponents (e + 127), one byte per key
//   [4112, 4128)  V scale exponents
// A stored value is code * 2^e; code * 2^e is exact in bf16, so the kernels
// convert codes to bf16 unscaled and apply the scales to scores (K) and to
// probabilities (V).  The bf16 pool keeps its K tile [16][D] and V^T tile
// [D][16] per region.
#include "mtn_kernels.h"
#include "mtn_device.h"

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>

namespace mtn {
namespace {

// two E4M3 codes (bytes 0, 1 or 2, 3 of w) -> two bf16, exact
template <bool HI>
__device__ __forceinline__ uint32_t f8_bf16x2(uint32_t w) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HI));
}
// 2^(byte r of w - 127) as a float (stored exponents are in [1, 254])
__device__ __forceinline__ float f8_scale(uint32_t w, int r) {
    return __uint_as_float(((w >> (8 * r)) & 0xFFu) << 23);
}
typedef __attribute__((ext_vector_type(4))) short s16x4_t;
// The 16-key PV product: lane (m, g4) brings the 4 keys 4 g4 .. 4 g4 + 3 of
// both operands (the 16x16x16 MFMA's k slice of the lane).
__device__ __forceinline__ f32x4_t mfma_pv(const uint2 &a, const uint2 &b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, a),
                                                      __builtin_bit_cast(s16x4_t, b), c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// fused RoPE + quantize + append: one wave per (token, kv head); lane i holds
// the rotation pair (i, i + 64)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_append_fp8(PoolGeom g, PlanView p, int32_t layer,
                                                    const bf16_t *__restrict__ k,
                                                    const bf16_t *__restrict__ v) {
    const int lane = threadIdx.x & 63;
    const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (item >= (int64_t)p.n_tok * g.hkv) return;  // whole waves
    const int h = (int)(item % g.hkv);
    const int t = (int)(item / g.hkv);
    const int64_t row = p.tok_row[t];
    const bf16_t *kr = k + (row * g.hkv + h) * kF8D;
    const bf16_t *vr = v + (row * g.hkv + h) * kF8D;
    const float2 cs = p.rope[(int64_t)t * (kF8D / 2) + lane];
    const float x0 = to_f32(kr[lane]), x1 = to_f32(kr[lane + 64]);
    const float y0 = fmaf(x0, cs.x, -x1 * cs.y);
    const float y1 = fmaf(x1, cs.x, x0 * cs.y);
    const float v0 = to_f32(vr[lane]), v1 = to_f32(vr[lane + 64]);
    uint8_t *tile = (uint8_t *)g.kv + (int64_t)layer * g.layer_stride +
                    (int64_t)p.tok_block[t] * g.block_stride + (int64_t)h * g.head_stride;
    store_token_fp8(tile, p.tok_off[t], y0, y1, v0, v1, lane);
}

// ---------------------------------------------------------------------------
// MFMA decode attention over fp8 blocks (F8) or bf16 blocks, D = 128
// ---------------------------------------------------------------------------
// One work unit = (query token, kv head, split segment), one workgroup of NG
// waves; the unit's keys are cut into NG consecutive segments and each wave
// streams its own segment through its own LDS ring of NBUF blocks (no
// barrier inside the loop).  Per block, one wave computes all G heads:
//   S[key][head]  = K[key][:] . Q^T   four 16x16x32 MFMAs (A = K as bf16)
//   O^T[d][head] += V^T[d][key] . P'  eight 16x16x16 MFMAs (A = V as bf16)
// (fp8 codes convert to bf16 exactly; bf16 blocks are used as they are).
// Lane l (n = l % 16, g4 = l / 16) holds head n (heads >= G are zero
// queries): its QK B operand covers dims 32 g4 .. 32 g4 + 31, its scores are
// keys 4 g4 .. 4 g4 + 3, which is exactly its PV B operand, and its output
// accumulators are dims 32 g4 + 8 i + j (i < 4, j < 8) -- the PV MFMA j
// takes dims 8 m + j on its rows m.  The online softmax keeps a per-head
// reference max that moves only when a block's max exceeds it by more than
// 2^8, so the accumulator rescale is rare.  At the end the waves' (max, sum,
// acc) are merged through LDS by log-sum-exp.
// Launch shape, from sweeps of waves per workgroup (2..8) and ring depth
// (2..4) at the 128-session G = 8 (512 units per launch), 64-session G = 1
// and 256-session G = 4 (2048 units) shapes: two-block rings win everywhere;
// 4 waves win at G = 8 (fp8 5.97 TB/s against 5.86 with 8; bf16 6.63 against
// 6.59), 8 waves at the smaller groups (fp8 6.14-6.21 against 5.79-5.95).
template <bool F8, int G>
struct MfmaShape {
#ifdef MTN_MFMA_GROUPS
    static constexpr int NG = MTN_MFMA_GROUPS;
#else
    static constexpr int NG = G >= 8 ? 4 : 8;
#endif
#ifdef MTN_MFMA_NBUF
    static constexpr int NBUF = MTN_MFMA_NBUF;
#else
    static constexpr int NBUF = 2;
#endif
};

template <bool F8, int G, int NG, int NBUF>
__global__ __launch_bounds__(64 * NG) void k_attn_mfma(AttnArgs a) {
    constexpr int D = kF8D;
    // one block's ring slot: fp8 codes + exponents, or the bf16 K and V^T tiles
    constexpr int BLK = F8 ? kF8Read : 2 * kBlock * D * 2;
    // DMA instructions per block: 4 x 1 KiB + the 32 exponent bytes, or 8 x 1 KiB
    constexpr int NIW = F8 ? 5 : 8;
    constexpr int ESZ = F8 ? 1 : 2;  // bytes per stored element
    static_assert(G >= 1 && G <= 16, "heads per kv group");
    static_assert(NBUF >= 2 && NBUF <= 8, "ring depth");
    static_assert(NBUF * BLK >= 16 * D * 4, "merge scratch fits one wave's ring");
    __shared__ __attribute__((aligned(16))) uint8_t ring[NG][NBUF][BLK];
    __shared__ float sM[NG][16], sL[NG][16];

    const int lane = threadIdx.x & 63;
    const int n = lane & 15, g4 = lane >> 4;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const PoolGeom &g = a.g;
    const uint32_t ns = (uint32_t)a.n_split;
    const UnitIdx ui = decode_unit(blockIdx.x, ns, (uint32_t)g.hkv);
    const int split = ui.split, kvh = ui.kvh, t = ui.t;
    const int sid = __builtin_amdgcn_readfirstlane(a.p.tok_sid[t]);
    const int pos = __builtin_amdgcn_readfirstlane(a.p.tok_pos[t]);
    const int64_t row = __builtin_amdgcn_readfirstlane(a.p.tok_row[t]);
    // With a fused append, the wave holding the unit's last segment (which
    // ends at the query's own position) takes the newest key and value from
    // the inputs: it writes their stored form into its LDS copy of the last
    // block, at the token's slot, and into the pool after its last barrier.
    const bool own_new = a.k_new != nullptr && split == a.n_split - 1 && wv == NG - 1;

    const VisRange vr = vis_range(g, pos);
    const int nv = vr.n_sb + vr.n_rb;
    const uint32_t nseg = ns * NG, seg = (uint32_t)split * NG + wv;
    const int v0 = __builtin_amdgcn_readfirstlane(seg_begin(seg, nseg, nv));
    const int v1 = __builtin_amdgcn_readfirstlane(seg_begin(seg + 1, nseg, nv));
    const int nblk = v1 - v0;
    const uint8_t *head_base = g.kv + (int64_t)a.layer * g.layer_stride + (int64_t)kvh * g.head_stride;
    const int32_t *trow = g.table + (int64_t)sid * g.row_len;
    const uint32_t ring0 = lds_addr(&ring[wv][0][0]);

    BlockIter it_issue(g, vr, v0), it_proc(g, vr, v0);
    auto issue = [&](int i) {
        int lb, lo, hi;
        it_issue.get(&lb, &lo, &hi);
        it_issue.next();
        int phys = scalar_ld(trow, __builtin_amdgcn_readfirstlane(lb));
        phys = phys < 0 ? 0 : phys;  // unassigned: any valid block, every slot masked
        const uint8_t *src = head_base + (int64_t)phys * g.block_stride;
        const uint32_t dst = ring0 + (uint32_t)((i % NBUF) * BLK);
        if constexpr (F8) {
#pragma unroll
            for (int j = 0; j < 4; ++j) dma16(src + swz(j * 64 + lane) * 16, dst + j * 1024);
            if (lane < 2) dma16(src + kF8Exp + lane * 16, dst + kF8Exp);
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) dma16(src + swz(j * 64 + lane) * 16, dst + j * 1024);
        }
    };
    const int pre = nblk < NBUF - 1 ? nblk : NBUF - 1;
    for (int i = 0; i < pre; ++i) issue(i);

    // ---- q prologue: rotate at pos, fold the softmax scale (log2 domain);
    // the B operand of QK MFMA s holds dims 32 g4 + 8 s .. + 7 of head n.
    const int d0 = 32 * g4;
    const int dp = d0 ^ 64;  // RoPE partner dims
    uint4 qb[4];
    const float2 *rp = a.p.rope + (int64_t)t * (D / 2) + (d0 & 63);
    const float sgn = g4 < 2 ? -1.f : 1.f;
    {
        const bool hv = n < G;
        const bf16_t *qh = (const bf16_t *)a.q + (row * g.hq + (int64_t)kvh * G + (hv ? n : 0)) * D;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            float x[8], y[8];
            unpack8(((const uint4 *)(qh + d0))[s], x);
            unpack8(((const uint4 *)(qh + dp))[s], y);
            uint32_t w[4];
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
                const float2 c0 = rp[8 * s + e], c1 = rp[8 * s + e + 1];
                const float r0 = fmaf(x[e], c0.x, sgn * y[e] * c0.y) * a.scale_log2;
                const float r1 = fmaf(x[e + 1], c1.x, sgn * y[e + 1] * c1.y) * a.scale_log2;
                w[e / 2] = hv ? pack_bf16x2(r0, r1) : 0u;
            }
            qb[s] = make_uint4(w[0], w[1], w[2], w[3]);
        }
    }
    // The owner rotates (and, fp8, quantizes) the newest key and value two
    // dims per lane (dims d0 + 2 n, d0 + 2 n + 1), exactly as the append
    // kernel does.
    uint32_t kc2 = 0, vc2 = 0;
    int ek_new = 0, ev_new = 0;
    const int dd = d0 + 2 * n;
    if (own_new) {
        const bf16_t *kh = (const bf16_t *)a.k_new + (row * g.hkv + kvh) * D;
        const bf16_t *vh = (const bf16_t *)a.v_new + (row * g.hkv + kvh) * D;
        const uint32_t kx = *(const uint32_t *)(kh + dd), ky = *(const uint32_t *)(kh + (dd ^ 64));
        const uint32_t vx = *(const uint32_t *)(vh + dd);
        const float4 cs = *(const float4 *)(rp + 2 * n);  // (cos, sin) of dims dd, dd + 1
        // rotated exactly as the append kernel does
        const float k0 = fmaf(__uint_as_float(kx << 16), cs.x, sgn * __uint_as_float(ky << 16) * cs.y);
        const float k1 = fmaf(__uint_as_float(kx & 0xFFFF0000u), cs.z,
                              sgn * __uint_as_float(ky & 0xFFFF0000u) * cs.w);
        if constexpr (F8) {
            const float v0 = __uint_as_float(vx << 16), v1 = __uint_as_float(vx & 0xFFFF0000u);
            float ak = fmaxf(fabsf(k0), fabsf(k1)), av = fmaxf(fabsf(v0), fabsf(v1));
#pragma unroll
            for (int m = 1; m < 16; m <<= 1) {  // the 16 lanes of a row, then the rows
                ak = fmaxf(ak, __shfl_xor(ak, m, 64));
                av = fmaxf(av, __shfl_xor(av, m, 64));
            }
            ek_new = __builtin_amdgcn_readfirstlane(f8_scale_exp(rows_max(ak)));
            ev_new = __builtin_amdgcn_readfirstlane(f8_scale_exp(rows_max(av)));
            kc2 = f8_pack<false>(ldexpf(k0, -ek_new), ldexpf(k1, -ek_new), 0u);
            vc2 = f8_pack<false>(ldexpf(v0, -ev_new), ldexpf(v1, -ev_new), 0u);
        } else {
            kc2 = pack_bf16x2(k0, k1);  // rounded to the stored type as the append does
            vc2 = vx;
        }
    }
    const int toff = __builtin_amdgcn_readfirstlane(a.p.tok_off[t]);  // the newest key's slot
    // the newest token's stored bytes into a ring slot holding its block (the
    // slot's DMA has landed); chunk x of the block lives at swz(x)
    auto put_new = [&](uint8_t *blk) {
        auto at = [&](int byte) { return blk + swz(byte >> 4) * 16 + (byte & 15); };
        if constexpr (F8) {
            *(uint16_t *)at(toff * D + dd) = (uint16_t)kc2;
            const int vb = kF8Tile + ((toff >> 2) * D + dd) * 4 + (toff & 3);
            *at(vb) = (uint8_t)vc2;
            *at(vb + 4) = (uint8_t)(vc2 >> 8);
            if (lane == 0) {
                blk[kF8Exp + toff] = (uint8_t)(ek_new + 127);
                blk[kF8Exp + kBlock + toff] = (uint8_t)(ev_new + 127);
            }
        } else {
            *(uint32_t *)at((toff * D + dd) * 2) = kc2;
            const int vb = kBlock * D * 2 + (dd * kBlock + toff) * 2;  // V^T [D][16]
            *(uint16_t *)at(vb) = (uint16_t)vc2;
            *(uint16_t *)at(vb + kBlock * 2) = (uint16_t)(vc2 >> 16);
        }
        wave_sync();
    };

    float m_ref = -INFINITY, lsum = 0.f;
    f32x4_t acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // per-lane LDS offsets of the K and V fragments inside a ring slot (the
    // chunk swizzle keeps each 16-lane read phase on 16 distinct bank groups)
    //   fp8:  K chunks 8 n + 2 g4 (+1); V quads chunks 128 + 32 g4 + 2 n (+1)
    //   bf16: K chunks 16 n + 4 g4 + s; V^T row 8 n + j, keys 4 g4 .. + 3 at
    //         chunk 256 + 2 (8 n + j) + g4 / 2, byte 8 (g4 % 2)
    const int ko0 = F8 ? swz(8 * n + 2 * g4) * 16 : 0, ko1 = F8 ? swz(8 * n + 2 * g4 + 1) * 16 : 0;
    const int vo0 = F8 ? swz(128 + 32 * g4 + 2 * n) * 16 : 0;
    const int vo1 = F8 ? swz(128 + 32 * g4 + 2 * n + 1) * 16 : 0;

    for (int i = 0; i < nblk; ++i) {
        // block i has landed once at most the blocks issued after it are in flight
        vm_wait_blocks<NIW, NBUF - 2>(min(NBUF - 2, nblk - 1 - i));
        if (i + NBUF - 1 < nblk) issue(i + NBUF - 1);
        const uint8_t *blk = &ring[wv][i % NBUF][0];
        int lb, lo, hi;
        it_proc.get(&lb, &lo, &hi);
        it_proc.next();
        if (scalar_ld(trow, __builtin_amdgcn_readfirstlane(lb)) < 0) hi = lo;  // unassigned
        if (own_new && i == nblk - 1) put_new((uint8_t *)blk);  // slot hi - 1 is the newest key
        const bool full = lo == 0 && hi == kBlock;

        // QK: S[key][head] for keys 4 g4 + r, head n
        f32x4_t c = {0.f, 0.f, 0.f, 0.f};
        uint2 vw2[8];  // PV A operands (4 keys of dim 8 n + j), bf16 pool
        uint32_t vw[8];  // the same as fp8 codes
        uint32_t evs = 0;
        float sc[4];
        if constexpr (F8) {
            const uint4 k0 = *(const uint4 *)(blk + ko0);
            const uint4 k1 = *(const uint4 *)(blk + ko1);
            const uint4 w0 = *(const uint4 *)(blk + vo0);
            const uint4 w1 = *(const uint4 *)(blk + vo1);
            const uint32_t eks = *(const uint32_t *)(blk + kF8Exp + 4 * g4);
            evs = *(const uint32_t *)(blk + kF8Exp + kBlock + 4 * g4);
            const uint32_t kw[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const uint4 af = make_uint4(f8_bf16x2<false>(kw[2 * s]), f8_bf16x2<true>(kw[2 * s]),
                                            f8_bf16x2<false>(kw[2 * s + 1]), f8_bf16x2<true>(kw[2 * s + 1]));
                c = mfma16x16x32(af, qb[s], c);
            }
            vw[0] = w0.x; vw[1] = w0.y; vw[2] = w0.z; vw[3] = w0.w;
            vw[4] = w1.x; vw[5] = w1.y; vw[6] = w1.z; vw[7] = w1.w;
#pragma unroll
            for (int r = 0; r < 4; ++r) sc[r] = c[r] * f8_scale(eks, r);
        } else {
#pragma unroll
            for (int s = 0; s < 4; ++s)
                c = mfma16x16x32(*(const uint4 *)(blk + swz(16 * n + 4 * g4 + s) * 16), qb[s], c);
#pragma unroll
            for (int j = 0; j < 8; ++j)
                vw2[j] = *(const uint2 *)(blk + swz(256 + 16 * n + 2 * j + (g4 >> 1)) * 16 + 8 * (g4 & 1));
#pragma unroll
            for (int r = 0; r < 4; ++r) sc[r] = c[r];
        }
        if (!full) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int key = 4 * g4 + r;
                sc[r] = (key >= lo && key < hi) ? sc[r] : -INFINITY;
            }
        }
        const float mx = rows_max(vmax3(vmax3(sc[0], sc[1], sc[2]), sc[3], sc[0]));
        const bool bump = mx > m_ref + 8.f;
        if (__builtin_amdgcn_ballot_w64(bump)) {
            const float mnew = bump ? mx : m_ref;
            const float alpha = mnew == m_ref ? 1.f : __builtin_amdgcn_exp2f(m_ref - mnew);
            m_ref = mnew;
            lsum *= alpha;
#pragma unroll
            for (int j = 0; j < 8; ++j) acc[j] *= alpha;
        }
        const float mr = m_ref == -INFINITY ? 0.f : m_ref;
        float pv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) pv[r] = __builtin_amdgcn_exp2f(sc[r] - mr);
        lsum += (pv[0] + pv[1]) + (pv[2] + pv[3]);
        if constexpr (F8) {
            // fold the value scales into the probabilities
#pragma unroll
            for (int r = 0; r < 4; ++r) pv[r] *= f8_scale(evs, r);
        }
        if (!full) {
            // invisible slots: zero probability, and zero values (they may be NaN)
            uint32_t bm = 0;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int key = 4 * g4 + r;
                const bool ok = key >= lo && key < hi;
                pv[r] = ok ? pv[r] : 0.f;
                bm |= ok ? (0xFFu << (8 * r)) : 0u;
            }
            if constexpr (F8) {
#pragma unroll
                for (int j = 0; j < 8; ++j) vw[j] &= bm;
            } else {
                // bf16 keys: two bytes of the mask per key
                const uint32_t m01 = (bm & 0x1u ? 0x0000FFFFu : 0u) | (bm & 0x100u ? 0xFFFF0000u : 0u);
                const uint32_t m23 = (bm & 0x10000u ? 0x0000FFFFu : 0u) | (bm & 0x1000000u ? 0xFFFF0000u : 0u);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    vw2[j].x &= m01;
                    vw2[j].y &= m23;
                }
            }
        }
        const uint2 pb = make_uint2(pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]));
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if constexpr (F8)
                acc[j] = mfma_pv(make_uint2(f8_bf16x2<false>(vw[j]), f8_bf16x2<true>(vw[j])), pb, acc[j]);
            else
                acc[j] = mfma_pv(vw2[j], pb, acc[j]);
        }
    }

    float L = rows_sum(lsum);

    // the pool copy of the newest key and value, for later launches; issued
    // after the wave's last barrier (a barrier's release fence would wait for
    // these scattered stores)
    auto store_new = [&]() {
        const int64_t tb = __builtin_amdgcn_readfirstlane(a.p.tok_block[t]);
        uint8_t *tile = (uint8_t *)g.kv + (int64_t)a.layer * g.layer_stride + tb * g.block_stride +
                        (int64_t)kvh * g.head_stride;
        if constexpr (F8) {
            *(uint16_t *)(tile + toff * D + dd) = (uint16_t)kc2;  // K row bytes dd, dd + 1
            uint8_t *vq = tile + kF8Tile + (toff >> 2) * (4 * D) + (toff & 3);
            vq[dd * 4] = (uint8_t)vc2;
            vq[(dd + 1) * 4] = (uint8_t)(vc2 >> 8);
            if (lane == 0) {
                tile[kF8Exp + toff] = (uint8_t)(ek_new + 127);
                tile[kF8Exp + kBlock + toff] = (uint8_t)(ev_new + 127);
            }
        } else {
            *(uint32_t *)(tile + (toff * D + dd) * 2) = kc2;  // K row elements dd, dd + 1
            uint16_t *vt = (uint16_t *)(tile + g.tile_bytes);  // V^T [D][16]
            vt[dd * kBlock + toff] = (uint16_t)vc2;
            vt[(dd + 1) * kBlock + toff] = (uint16_t)(vc2 >> 16);
        }
    };

    const int hq0 = kvh * G;
    if constexpr (NG > 1) {
        // every wave hands (m, l, acc) over through its own drained ring; then
        // all threads of the workgroup merge them by log-sum-exp, one pair of
        // output dims per thread and step (a wave covers one head's row)
        float *scr = (float *)&ring[wv][0][0] + n * D + d0;  // [16][D]
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            *(float4 *)(scr + 8 * i) = make_float4(acc[0][i], acc[1][i], acc[2][i], acc[3][i]);
            *(float4 *)(scr + 8 * i + 4) = make_float4(acc[4][i], acc[5][i], acc[6][i], acc[7][i]);
        }
        if (g4 == 0) {
            sM[wv][n] = m_ref;
            sL[wv][n] = L;
        }
        __syncthreads();
        if (own_new) store_new();
        for (int e = threadIdx.x; e < G * (D / 2); e += 64 * NG) {
            const int h = e / (D / 2), d = 2 * (e % (D / 2));
            float M = sM[0][h];
#pragma unroll
            for (int q = 1; q < NG; ++q) M = fmaxf(M, sM[q][h]);
            const float Mn = M == -INFINITY ? 0.f : M;
            float l = 0.f, o0 = 0.f, o1 = 0.f;
#pragma unroll
            for (int q = 0; q < NG; ++q) {
                const float wq = __builtin_amdgcn_exp2f(sM[q][h] - Mn);
                const float2 x = *(const float2 *)((const float *)&ring[q][0][0] + h * D + d);
                l = fmaf(sL[q][h], wq, l);
                o0 = fmaf(wq, x.x, o0);
                o1 = fmaf(wq, x.y, o1);
            }
            if (a.n_split == 1) {
                const float inv = 1.f / l;
                *(uint32_t *)((bf16_t *)a.out + (row * g.hq + hq0 + h) * D + d) = pack_bf16x2(o0 * inv, o1 * inv);
                if (a.lse && d == 0)
                    a.lse[row * g.hq + hq0 + h] = (M + __builtin_amdgcn_logf(l)) * 0.6931471805599453f;
            } else {
                const int64_t base = ((int64_t)t * g.hq + hq0 + h) * ns + split;
                *(float2 *)(a.part + base * D + d) = make_float2(o0, o1);
                if (d == 0) {
                    float *pml = a.part + (int64_t)a.p.n_tok * g.hq * ns * D;
                    pml[base * 2] = M;
                    pml[base * 2 + 1] = l;
                }
            }
        }
    } else {
        if (n < G) {
            if (a.n_split == 1) {
                const float inv = 1.f / L;
                bf16_t *ob = (bf16_t *)a.out + (row * g.hq + hq0 + n) * D + d0;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    *(uint4 *)(ob + 8 * i) =
                        make_uint4(pack_bf16x2(acc[0][i] * inv, acc[1][i] * inv),
                                   pack_bf16x2(acc[2][i] * inv, acc[3][i] * inv),
                                   pack_bf16x2(acc[4][i] * inv, acc[5][i] * inv),
                                   pack_bf16x2(acc[6][i] * inv, acc[7][i] * inv));
                if (a.lse && g4 == 0)
                    a.lse[row * g.hq + hq0 + n] = (m_ref + __builtin_amdgcn_logf(L)) * 0.6931471805599453f;
            } else {
                const int64_t base = ((int64_t)t * g.hq + hq0 + n) * ns + split;
                float *pacc = a.part + base * D + d0;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    *(float4 *)(pacc + 8 * i) = make_float4(acc[0][i], acc[1][i], acc[2][i], acc[3][i]);
                    *(float4 *)(pacc + 8 * i + 4) = make_float4(acc[4][i], acc[5][i], acc[6][i], acc[7][i]);
                }
                if (g4 == 0) {
                    float *pml = a.part + (int64_t)a.p.n_tok * g.hq * ns * D;
                    pml[base * 2] = m_ref;
                    pml[base * 2 + 1] = L;
                }
            }
        }
        if (own_new) store_new();  // one wave: it owns the newest key
    }
}

// ---------------------------------------------------------------------------
// debug poison: NaN codes and infinite scales into every slot whose live bit
// is clear
// ---------------------------------------------------------------------------
__global__ void k_poison_fp8(PoolGeom g, int32_t n_layers, int64_t n_blocks,
                             const uint16_t *__restrict__ live) {
    const int64_t n_items = (int64_t)n_layers * n_blocks * g.hkv;
    for (int64_t it = blockIdx.x; it < n_items; it += gridDim.x) {
        const int h = (int)(it % g.hkv);
        const int64_t b = (it / g.hkv) % n_blocks;
        const int l = (int)(it / ((int64_t)g.hkv * n_blocks));
        const uint16_t lm = live[b];
        if (lm == 0xFFFF) continue;
        uint8_t *tile = (uint8_t *)g.kv + (int64_t)l * g.layer_stride + b * g.block_stride +
                        (int64_t)h * g.head_stride;
        for (int e = threadIdx.x; e < kF8Tile; e += blockDim.x) {
            const int key = e / kF8D, d = e % kF8D;
            if (!((lm >> key) & 1)) {
                tile[e] = 0x7F;
                tile[kF8Tile + ((key >> 2) * kF8D + d) * 4 + (key & 3)] = 0x7F;
            }
        }
        if (threadIdx.x < 2 * kBlock) {
            const int key = threadIdx.x % kBlock;
            if (!((lm >> key) & 1)) tile[kF8Exp + threadIdx.x] = 0xFF;
        }
    }
}

template <bool F8, int G>
hipError_t launch_mfma_g(const AttnArgs &a, hipStream_t s) {
    using S = MfmaShape<F8, G>;
    const int64_t units = (int64_t)a.p.n_tok * a.g.hkv * a.n_split;
    if (units == 0) return hipSuccess;
    if (units > INT32_MAX) return hipErrorInvalidValue;  // one grid dimension, 32-bit unit index
    hipLaunchKernelGGL((k_attn_mfma<F8, G, S::NG, S::NBUF>), dim3((unsigned)units), dim3(64 * S::NG),
                       0, s, a);
    return hipGetLastError();
}
template <bool F8, int G>
int resident_mfma_g() {
    using S = MfmaShape<F8, G>;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_attn_mfma<F8, G, S::NG, S::NBUF>,
                                                     64 * S::NG, 0) != hipSuccess)
        return 1;
    // The split rule fills these slots.  It counts the workgroups whose rings
    // hold about 64 KiB of copies in flight per CU (bf16: one of 4 waves x 2
    // blocks x 8 KiB; fp8: two of 4 x 2 x 4128 bytes), not the occupancy
    // limit.  Measured per launch with the split merge, 128 units (32
    // sessions, G = 8): bf16 49.7 us at split 2 against 52.1 at 4, fp8 32.4
    // at split 4 against 37.7 at 2; 256 units: bf16 87.2 unsplit against 93.2
    // at split 2, fp8 53.7 at split 2 against 60.8 unsplit.  (With more
    // streams in flight the decode ran slower: deeper rings, more waves per
    // unit, and fp8 split to fill the four workgroups its registers allow.)
    constexpr int kRing = S::NG * S::NBUF * (F8 ? kF8Read : 2 * kBlock * kF8D * 2);
    constexpr int kTarget = ((64 << 10) + kRing / 2) / kRing;
    return std::min(std::max(n, 1), std::max(kTarget, 1));
}
template <bool F8>
hipError_t launch_mfma(const AttnArgs &a, hipStream_t s) {
    switch (a.g.hq / a.g.hkv) {
        case 1: return launch_mfma_g<F8, 1>(a, s);
        case 2: return launch_mfma_g<F8, 2>(a, s);
        case 4: return launch_mfma_g<F8, 4>(a, s);
        default: return launch_mfma_g<F8, 8>(a, s);
    }
}
template <bool F8>
int resident_mfma(int g) {
    switch (g) {
        case 1: return resident_mfma_g<F8, 1>();
        case 2: return resident_mfma_g<F8, 2>();
        case 4: return resident_mfma_g<F8, 4>();
        default: return resident_mfma_g<F8, 8>();
    }
}

}  // namespace

int fp8_head_stride(int d) {
    // codes + exponents, rounded up to 128 bytes so every region starts on a
    // line boundary
    return d == kF8D ? ((kF8Read + 127) / 128) * 128 : 0;
}

bool attn_fp8_supported(int d, int g) {
    return d == kF8D && (g == 1 || g == 2 || g == 4 || g == 8);
}

int attn_fp8_resident_per_cu(int g) { return resident_mfma<true>(g); }

bool attn_mfma_bf16_supported(int d, int g) { return attn_fp8_supported(d, g); }
int attn_mfma_bf16_resident_per_cu(int g) { return resident_mfma<false>(g); }
hipError_t launch_attn_mfma_bf16(const AttnArgs &a, hipStream_t s) {
    if (!attn_mfma_bf16_supported(a.g.d, a.g.hq / a.g.hkv)) return hipErrorInvalidValue;
    return launch_mfma<false>(a, s);
}

hipError_t launch_append_fp8(const PoolGeom &g, const PlanView &p, int32_t layer, const void *k,
                             const void *v, hipStream_t s) {
    if (g.d != kF8D) return hipErrorInvalidValue;
    const int64_t waves = (int64_t)p.n_tok * g.hkv;
    if (waves == 0) return hipSuccess;
    hipLaunchKernelGGL(k_append_fp8, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s, g, p, layer,
                       (const bf16_t *)k, (const bf16_t *)v);
    return hipGetLastError();
}

hipError_t launch_attn_fp8(const AttnArgs &a, hipStream_t s) {
    if (!attn_fp8_supported(a.g.d, a.g.hq / a.g.hkv)) return hipErrorInvalidValue;
    return launch_mfma<true>(a, s);
}

hipError_t launch_poison_fp8(const PoolGeom &g, int32_t n_layers, int64_t n_blocks,
                             const uint16_t *live, hipStream_t s) {
    hipLaunchKernelGGL(k_poison_fp8, dim3(8192), dim3(256), 0, s, g, n_layers, n_blocks, live);
    return hipGetLastError();
}

}  // namespace mtn
