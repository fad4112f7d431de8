// Internal launch interface between the host library (mtn_host.cpp) and the
// gfx950 kernels (mtn_kernels.hip).  Not part of the public C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mtn {

// Geometry of the paged pool as the kernels see it.  Byte strides; the pool
// layout is [layer][block][kv_head]{K tile [16][D], V^T tile [D][16]}.
struct PoolGeom {
    const uint8_t *kv;       // pool base (device)
    int64_t layer_stride;    // bytes per layer
    int64_t block_stride;    // bytes per (layer, block)
    int64_t head_stride;     // bytes per (layer, block, kv head) = 2 tiles
    int64_t tile_bytes;      // bytes of one K (or V^T) tile
    const int32_t *table;    // [max_sessions][row_len] physical block ids
    int32_t row_len;
    int32_t n_sink;          // S (0 when unbounded)
    int32_t window;          // W, or -1 when unbounded
    int32_t ring;            // R tokens (unbounded: row_len * 16)
    int32_t n_sink_blocks;   // ceil(S / 16)
    int32_t hq, hkv, d;
};

// One planned token: which session, absolute position, io row, slot.
struct PlanView {
    const int32_t *tok_sid;
    const int32_t *tok_pos;
    const int32_t *tok_row;
    const int32_t *tok_block;
    const int32_t *tok_off;
    const float2  *rope;     // [T][D/2] (cos, sin) of pos * theta^(-2i/D)
    int32_t n_tok;
};

struct AttnArgs {
    PoolGeom g;
    PlanView p;
    int32_t layer;
    const void *q;           // [rows][Hq][D], row = tok_row[t]
    void *out;               // [rows][Hq][D]
    float *lse;              // [rows][Hq] or null
    float *part;             // split partials (acc [unit][G][D] then ml [unit][G][2])
    int32_t n_split;
    float scale_log2;        // softmax scale * log2(e)
    const uint8_t *zero_page;  // 16 KiB of zeros (DMA source of absent blocks)
    // decode with a fused append (or null): [rows][Hkv][D] keys / values of
    // the planned tokens, each the newest position of its own query
    const void *k_new;
    const void *v_new;
};

// dtype codes match the public MTN_F32 / MTN_BF16 / MTN_FP8_E4M3
hipError_t launch_plan_apply(const int32_t *upd_idx, const int32_t *upd_val, int32_t n_upd,
                             int32_t *table, const int32_t *tok_pos, int32_t n_tok,
                             const double *inv_freq, int32_t half_d, float2 *rope,
                             hipStream_t s);

// Append (fp32 / bf16 pools) over runs: run r covers planned tokens
// run_tok0[r] .. + run_len[r] - 1, consecutive slots of one block.
hipError_t launch_append(int dtype, const PoolGeom &g, const PlanView &p, int32_t layer,
                         const void *k, const void *v, const int32_t *run_tok0,
                         const int32_t *run_len, int32_t n_runs, hipStream_t s);

// Vector (VALU) attention over items = planned tokens: decode, and the fp32
// chunk prefill.  Returns hipErrorInvalidValue for shapes with no instance.
hipError_t launch_attn_valu(int dtype, const AttnArgs &a, hipStream_t s);
hipError_t launch_merge(int dtype, const AttnArgs &a, hipStream_t s);

// MFMA chunk-prefill attention (bf16 or fp8 pool, D = 128): one workgroup per (sequence,
// row pass, kv head).  items: n_items records of kPfItem int32 (32-byte
// aligned), one per row pass: {pass, first planned token t0, tokens, session
// id, position of t0, io row of t0, 0, 0}; token t0 + j of the sequence uses
// io row (row of t0) + j (multi-token plans always do); pass p covers the
// sequence's query rows [p, p + 1) * pass_rows (rows are token * G + group
// head).  pass_rows: prefill_rows_per_pass() or, to spread few sequences over
// more workgroups, 128 (prefill_pass_rows_valid).  zero_page: 16 KiB of
// device zeros, the DMA source of blocks a pass does not see.  a.k_new /
// a.v_new (both or neither; fp8 pool only; [rows][Hkv][D] bf16): the launch
// also appends the planned tokens (RoPE on K, quantized), which the caller may
// ask for only when every sequence takes exactly one row pass.
constexpr int kPfItem = 8;
int prefill_rows_per_pass();
bool prefill_pass_rows_valid(int rows);
hipError_t launch_prefill_mfma(int dtype, const AttnArgs &a, const int32_t *items, int32_t n_items,
                               int32_t pass_rows, const uint8_t *zero_page, hipStream_t s);

hipError_t launch_poison(int dtype, const PoolGeom &g, int32_t n_layers, int64_t n_blocks,
                         const uint16_t *live_mask, hipStream_t s);

hipError_t launch_copy(const void *src, void *dst, size_t bytes, hipStream_t s);
// streaming read of the whole 8 KiB chunks of `bytes` into LDS (nothing
// computed or written)
hipError_t launch_read(const void *src, size_t bytes, uint32_t *out, hipStream_t s);

// The library's static device workspace for split partials (a file-scope
// array, no allocation): its address on the current device and its size in
// floats.
hipError_t scratch_buffer(float **ptr, size_t *floats);

// FP8 (E4M3) KV cache, D = 128, bf16 io: bytes per (layer, block, kv head)
// region (0 for an unsupported head dim), the fused RoPE + quantize + append,
// the MFMA decode (k_new / v_new in AttnArgs select the fused append) and the
// debug poison.
int fp8_head_stride(int d);
bool attn_fp8_supported(int d, int g);
int attn_fp8_resident_per_cu(int g);
hipError_t launch_append_fp8(const PoolGeom &g, const PlanView &p, int32_t layer, const void *k,
                             const void *v, hipStream_t s);
hipError_t launch_attn_fp8(const AttnArgs &a, hipStream_t s);
hipError_t launch_poison_fp8(const PoolGeom &g, int32_t n_layers, int64_t n_blocks,
                             const uint16_t *live_mask, hipStream_t s);

// The same MFMA decode over bf16 blocks (D = 128, bf16 io), append fusable.
bool attn_mfma_bf16_supported(int d, int g);
int attn_mfma_bf16_resident_per_cu(int g);
hipError_t launch_attn_mfma_bf16(const AttnArgs &a, hipStream_t s);

bool attn_valu_supported(int dtype, int d, int g);
// workgroups of the vector attention kernel resident per CU (occupancy query)
int attn_valu_resident_per_cu(int dtype, int d, int g);
bool prefill_mfma_supported(int dtype, int d, int g);

constexpr int kBlock = 16;      // tokens per KV block
constexpr int kMaxSplit = 64;   // decode split cap

}  // namespace mtn
