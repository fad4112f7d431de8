// Device-side helpers shared by the gfx950 kernel sources of libmtn: element
// conversions, DPP / permlane reductions, the visible-range geometry of a
// query (sinks first, then the ring run), the LDS DMA primitives and the
// bf16 MFMA wrapper.  Included by the .hip sources only.
#pragma once
#include "mtn_kernels.h"

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace mtn {
namespace {

// FP8 KV region of one (layer, block, kv head), D = 128: K codes [16][128],
// V codes in key quads, then 16 K and 16 V scale-exponent bytes
constexpr int kF8D = 128;                 // head dim of the fp8 path
constexpr int kF8Tile = kBlock * kF8D;    // bytes of one K (or V) code tile
constexpr int kF8Exp = 2 * kF8Tile;       // offset of the exponent bytes
constexpr int kF8Read = 2 * kF8Tile + 32; // bytes a kernel reads per (block, head)

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

// ---------------------------------------------------------------------------
// element helpers
// ---------------------------------------------------------------------------
struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) {
    return __uint_as_float((uint32_t)x.bits << 16);
}
template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) {
    return x;
}
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) {
    __bf16 b = (__bf16)x;  // round to nearest even (hardware cvt on gfx950)
    return bf16_t{__builtin_bit_cast(uint16_t, b)};
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    bf16x2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                           __builtin_bit_cast(bf16x2_t, b), c, false);
}

// DPP helpers (row = 16 lanes, quad = 4 lanes)
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                                         0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}
constexpr int kQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]
constexpr int kRowRor4 = 0x124;  // row_ror:4
constexpr int kRowRor8 = 0x128;  // row_ror:8
constexpr int kRowShr4 = 0x114;  // row_shr:4 (lane i takes lane i - 4 of its row)

__device__ __forceinline__ float shfl_xor_f(float x, int m) {
    return __shfl_xor(x, m, 64);
}

// Exchange between rows (16-lane groups) with the gfx950 permlane swaps.
// Given (a, a), v_permlane16_swap returns rows (0, 0, 2, 2) of a in its first
// result and rows (1, 1, 3, 3) in its second; v_permlane32_swap returns rows
// (0, 1, 0, 1) and (2, 3, 2, 3): combining the two reduces across the pair.
// Pure VALU, no LDS round trip.  Only the compiler builtins are used, never
// inline assembly: the swap reads both of its operands and writes both, and
// a VALU write of either operand needs wait states before the swap.  The
// compiler's hazard recognizer inserts those (and the MFMA-result wait states
// when an operand comes from a matrix instruction) only for instructions it
// sees; an inline-asm copy feeding the swap was invisible to it, and rows 1
// and 3 -- the rows a swap takes from its second operand -- then read a stale
// copy.
// 16 bytes of bf16 as 8 floats
__device__ __forceinline__ void unpack8(const uint4 &v, float *x) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 8; ++e)
        x[e] = __uint_as_float((e & 1) ? (w[e / 2] & 0xFFFF0000u) : (w[e / 2] << 16));
}

template <bool HALF>
__device__ __forceinline__ void row_swap(unsigned x, unsigned &a, unsigned &b) {
    if constexpr (HALF) {
        const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
        a = r[0];
        b = r[1];
    } else {
        const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
        a = r[0];
        b = r[1];
    }
}
template <bool SUM, bool HALF>
__device__ __forceinline__ float rows_pair(float x) {
    unsigned a, b;
    row_swap<HALF>(__builtin_bit_cast(unsigned, x), a, b);
    const float fa = __builtin_bit_cast(float, a), fb = __builtin_bit_cast(float, b);
    return SUM ? fa + fb : fmaxf(fa, fb);
}

// max / sum over the 16 lanes that share (lane & 3) -- i.e. over the 16 keys
// of a block for one quarter index
__device__ __forceinline__ float keys_max(float x) {
    x = fmaxf(x, dpp<kRowRor4>(x));
    x = fmaxf(x, dpp<kRowRor8>(x));
    x = rows_pair<false, false>(x);
    return rows_pair<false, true>(x);
}
__device__ __forceinline__ float keys_sum(float x) {
    x += dpp<kRowRor4>(x);
    x += dpp<kRowRor8>(x);
    x = rows_pair<true, false>(x);
    return rows_pair<true, true>(x);
}

__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---------------------------------------------------------------------------
// visible-range geometry of one query (sinks first, then the ring run)
// ---------------------------------------------------------------------------
struct VisRange {
    int sink_tokens;  // min(S, t+1)
    int n_sb;         // sink blocks read
    int first;        // ring slot of the first window position
    int ring_n;       // window positions (0 = none)
    int n_rb;         // ring blocks read (a block may appear twice on a wrap)
};

__device__ __forceinline__ VisRange vis_range(const PoolGeom &g, int t) {
    VisRange r;
    r.sink_tokens = min(g.n_sink, t + 1);
    r.n_sb = (r.sink_tokens + kBlock - 1) / kBlock;
    int a = g.window < 0 ? 0 : max(g.n_sink, t - g.window + 1);
    if (a <= t) {
        r.ring_n = t - a + 1;
        r.first = g.window < 0 ? a : (a - g.n_sink) % g.ring;
        r.n_rb = ((r.first % kBlock) + r.ring_n + kBlock - 1) / kBlock;
    } else {
        r.ring_n = 0;
        r.first = 0;
        r.n_rb = 0;
    }
    return r;
}

// Launch indices of the decode kernels, decoded in 32 bits: 64-bit divisions
// expand into long scalar sequences, which every wave of a CU would run back
// to back on the shared scalar unit before its first copy.
// unit = (t * hkv + kvh) * n_split + split
struct UnitIdx {
    int t, kvh, split;
};
__device__ __forceinline__ UnitIdx decode_unit(uint32_t unit, uint32_t n_split, uint32_t hkv) {
    const uint32_t th = unit / n_split;
    const uint32_t t = th / hkv;
    return UnitIdx{(int)t, (int)(th - t * hkv), (int)(unit - th * n_split)};
}
// first virtual block of key segment seg (of nseg) over nv blocks:
// floor(seg * nv / nseg), in 32 bits whenever the product fits
__device__ __forceinline__ int seg_begin(uint32_t seg, uint32_t nseg, int nv) {
    const uint64_t prod = (uint64_t)seg * (uint32_t)nv;
    if (prod <= 0xFFFFFFFFull) return (int)((uint32_t)prod / nseg);
    return (int)(prod / nseg);
}

// logical block and valid slot range [lo, hi) of virtual block v
__device__ __forceinline__ void vblock(const PoolGeom &g, const VisRange &r, int v, int *lb,
                                       int *lo, int *hi) {
    if (v < r.n_sb) {
        *lb = v;
        *lo = 0;
        *hi = min(kBlock, r.sink_tokens - v * kBlock);
        return;
    }
    int u = v - r.n_sb;
    int ring_blocks = g.ring / kBlock;
    *lb = g.n_sink_blocks + (r.first / kBlock + u) % ring_blocks;
    *lo = (u == 0) ? r.first % kBlock : 0;
    *hi = (u == r.n_rb - 1) ? ((r.first % kBlock) + r.ring_n - 1) % kBlock + 1 : kBlock;
}

// Walks the virtual blocks v0, v0 + 1, ... of one query without integer
// division inside the loop (one modulo at construction).
struct BlockIter {
    int v, n_sb, sink_tokens, n_rb, first_off, last_hi, rb, ring_blocks, nsb, rb_start;
    __device__ __forceinline__ BlockIter(const PoolGeom &g, const VisRange &r, int v0) {
        v = v0;
        n_sb = r.n_sb;
        sink_tokens = r.sink_tokens;
        n_rb = r.n_rb;
        first_off = r.first % kBlock;
        last_hi = r.ring_n > 0 ? (first_off + r.ring_n - 1) % kBlock + 1 : 0;
        ring_blocks = g.ring / kBlock;
        nsb = g.n_sink_blocks;
        rb_start = r.first / kBlock;
        rb = v0 > n_sb ? (rb_start + (v0 - n_sb)) % ring_blocks : rb_start;
    }
    __device__ __forceinline__ void get(int *lb, int *lo, int *hi) const {
        if (v < n_sb) {
            *lb = v;
            *lo = 0;
            *hi = min(kBlock, sink_tokens - v * kBlock);
        } else {
            const int u = v - n_sb;
            *lb = nsb + rb;
            *lo = (u == 0) ? first_off : 0;
            *hi = (u == n_rb - 1) ? last_hi : kBlock;
        }
    }
    __device__ __forceinline__ void next() {
        if (v >= n_sb) rb = (rb + 1 == ring_blocks) ? 0 : rb + 1;
        ++v;
    }
};

// Asynchronous 16-byte-per-lane copy global -> LDS (gfx950 LDS DMA).  Lane i
// of the wave writes LDS bytes [lds + 16 i, lds + 16 i + 16).  Issued from
// inline assembly so that the compiler does not guard later LDS reads with a
// full vmcnt(0); completion is awaited explicitly with vm_wait<N>().
// The M0 write and the load are one asm statement, with the wait state the
// hardware needs between an SALU write of M0 and an LDS DMA that reads it
// (the compiler inserts the same s_nop for its own LDS-DMA builtin).
// The K/V stream is read exactly once per launch: non-temporal ("nt") loads
// keep it from displacing reused lines in the caches (measured +2 % on the
// 128-session decode).
#ifndef MTN_DMA_POLICY
#define MTN_DMA_POLICY "nt"
#endif
__device__ __forceinline__ void dma16(const void *gptr, uint32_t lds) {
    asm volatile(
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %0, off " MTN_DMA_POLICY
        :
        : "v"(gptr), "s"(__builtin_amdgcn_readfirstlane(lds))
        : "memory", "m0");
}
// The same copy from a uniform 64-bit base held in SGPRs plus a 32-bit lane
// offset (the global "saddr" form): a stream whose base changes per block but
// whose lane offsets stay fixed needs no per-lane 64-bit address arithmetic.
// The base must be wave-uniform; it is read from the first lane so that it
// lives in SGPRs even where the compiler cannot prove it uniform.  The
// builtin returns int: each half goes through uint32_t, or a low word with
// bit 31 set would sign-extend into the high word.
// A wave-uniform 64-bit value rebuilt from its first lane's halves, so that
// it is held in SGPRs (each half goes through uint32_t: see dma16_s).
__device__ __forceinline__ uint64_t uniform64(uint64_t b) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    return (uint64_t)lo | ((uint64_t)hi << 32);
}
__device__ __forceinline__ void dma16_s(uint32_t voff, const void *sbase, uint32_t lds) {
    const uint64_t sb = uniform64((uint64_t)(uintptr_t)sbase);
    asm volatile(
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %0, %1 " MTN_DMA_POLICY
        :
        : "v"(voff), "s"(sb), "s"(__builtin_amdgcn_readfirstlane(lds))
        : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void vm_wait() {
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}
// wait until at most `after` blocks of NIW DMA instructions are outstanding
template <int NIW, int MAXA>
__device__ __forceinline__ void vm_wait_blocks(int after) {
    if constexpr (MAXA >= 6) { if (after >= 6) { vm_wait<6 * NIW>(); return; } }
    if constexpr (MAXA >= 5) { if (after == 5) { vm_wait<5 * NIW>(); return; } }
    if constexpr (MAXA >= 4) { if (after == 4) { vm_wait<4 * NIW>(); return; } }
    if constexpr (MAXA >= 3) { if (after == 3) { vm_wait<3 * NIW>(); return; } }
    if constexpr (MAXA >= 2) { if (after == 2) { vm_wait<2 * NIW>(); return; } }
    if constexpr (MAXA >= 1) { if (after == 1) { vm_wait<NIW>(); return; } }
    vm_wait<0>();
}
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}
// Read-only metadata (block table) fetched through the scalar unit: the
// table is never written while a kernel runs, so the constant address space
// is exact, and its loads are tracked apart from the vector-memory counter.
__device__ __forceinline__ int32_t scalar_ld(const int32_t *p, int idx) {
    return ((const __attribute__((address_space(4))) int32_t *)p)[idx];
}

// 16-byte chunk permutation of a block buffer: an involution that XORs the
// low four chunk bits with the next four, so every 16-byte read instruction of
// the ring (lane l takes chunk 4 l + c) spreads its lanes over all LDS banks.
// Chosen by measurement: 255 B/clk/CU of ds_read_b128 against 203 for a
// two-bit rotation and 117 unswizzled.
__device__ __forceinline__ int swz(int x) { return x ^ ((x >> 4) & 15); }

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

__device__ __forceinline__ f32x4_t mfma16x16x32(const uint4 &a, const uint4 &b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                    __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
// Maxima written as ordinary code, so that the compiler sees every read of
// a matrix-instruction result and spaces it as the hardware requires (inline
// assembly reading an MFMA accumulator is issued with no wait states).  Three
// operands map to one v_max3_f32.
__device__ __forceinline__ float vmax3(float a, float b, float c) {
    return fmaxf(fmaxf(a, b), c);
}
__device__ __forceinline__ float vmax2(float a, float b) { return fmaxf(a, b); }
// max over the four 16-lane rows (lanes with equal lane % 16)
__device__ __forceinline__ float rows_max(float x) {
    return rows_pair<false, true>(rows_pair<false, false>(x));
}
// smallest e with amax <= 448 * 2^e, clamped to [-126, 127]; 0 for amax = 0
__device__ __forceinline__ int f8_scale_exp(float amax) {
    if (!(amax > 0.f)) return 0;
    int e = __builtin_amdgcn_frexp_expf(amax) - 9;  // amax * 2^-e in [256, 512)
    if (ldexpf(amax, -e) > 448.f) ++e;
    return min(max(e, -126), 127);
}
// E4M3 codes of (a, b) into bytes 0, 1 (hi = false) or 2, 3 of `old`;
// round to nearest even, |a|, |b| <= 448
template <bool HI>
__device__ __forceinline__ uint32_t f8_pack(float a, float b, uint32_t old) {
    return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)old, HI);
}

// One token's K (already rotated) and V for one kv head into slot `off` of
// its pool region (D = 128), one wave: lane i holds dims i and i + 64 (the
// rotation pair).  fp8 pool: E4M3 codes under one power-of-two scale per row
// (K and V apart, from the row's largest magnitude), lane 0 writing the two
// exponent bytes.
__device__ __forceinline__ void store_token_fp8(uint8_t *region, int off, float k0, float k1,
                                                float v0, float v1, int lane) {
    float ak = fmaxf(fabsf(k0), fabsf(k1)), av = fmaxf(fabsf(v0), fabsf(v1));
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        ak = fmaxf(ak, __shfl_xor(ak, m, 64));
        av = fmaxf(av, __shfl_xor(av, m, 64));
    }
    const int ek = f8_scale_exp(ak), ev = f8_scale_exp(av);
    const uint32_t kc = f8_pack<false>(ldexpf(k0, -ek), ldexpf(k1, -ek), 0u);
    const uint32_t vc = f8_pack<false>(ldexpf(v0, -ev), ldexpf(v1, -ev), 0u);
    region[off * kF8D + lane] = (uint8_t)kc;
    region[off * kF8D + lane + 64] = (uint8_t)(kc >> 8);
    uint8_t *vq = region + kF8Tile + (off >> 2) * (4 * kF8D) + (off & 3);
    vq[lane * 4] = (uint8_t)vc;
    vq[(lane + 64) * 4] = (uint8_t)(vc >> 8);
    if (lane == 0) {
        region[kF8Exp + off] = (uint8_t)(ek + 127);
        region[kF8Exp + kBlock + off] = (uint8_t)(ev + 127);
    }
}

// sum over the four 16-lane rows (lanes with equal lane % 16)
__device__ __forceinline__ float rows_sum(float x) {
    return rows_pair<true, true>(rows_pair<true, false>(x));
}

}  // namespace
}  // namespace mtn
