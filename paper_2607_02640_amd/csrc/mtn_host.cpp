// Host side of libmtn: pool and session bookkeeping, the frame planner (block
// table, ring-slot map, eviction ranges, exhaustion checks), plan upload and
// kernel orchestration behind the C ABI declared in include/mtn.h.
//
// Method: Metronome (arXiv 2607.02640) §4.1 and App. A -- every session
// retains its first S tokens (pinned sink blocks, counted in the admission
// cap) and its last W tokens; §2 task model -- a frame prefills a chunk, then
// decodes single tokens, for all due sessions in one batch.
#include "mtn.h"
#include "mtn_kernels.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

using namespace mtn;

namespace {

constexpr int kStages = 4;  // pinned staging buffers in flight
constexpr size_t kZeroPage = 2 * kBlock * 128 * 4;  // 16 KiB

// Lowest-free-first block allocator over a bitmap (bit set = free).
class BlockAllocator {
  public:
    void reset(int64_t n) {
        n_ = n;
        words_.assign((size_t)((n + 63) / 64), ~0ull);
        if (n % 64) words_.back() = (1ull << (n % 64)) - 1;
        hint_ = 0;
        free_ = n;
    }
    int64_t n_free() const { return free_; }
    int64_t take() {  // caller checks n_free() > 0
        for (size_t w = hint_; w < words_.size(); ++w) {
            if (words_[w]) {
                int b = __builtin_ctzll(words_[w]);
                words_[w] &= words_[w] - 1;
                hint_ = w;
                --free_;
                return (int64_t)w * 64 + b;
            }
        }
        return -1;
    }
    void give(int64_t b) {
        words_[(size_t)(b / 64)] |= 1ull << (b % 64);
        hint_ = std::min(hint_, (size_t)(b / 64));
        ++free_;
    }
    bool is_free(int64_t b) const { return (words_[(size_t)(b / 64)] >> (b % 64)) & 1; }

  private:
    std::vector<uint64_t> words_;
    size_t hint_ = 0;
    int64_t n_ = 0, free_ = 0;
};

struct EventPair {
    hipEvent_t a, b;
};

}  // namespace

struct mtn_pool {
    mtn_pool_config cfg;
    bool host_only = false;
    bool unbounded = false;
    int S = 0, W = -1, R = 0, nsb = 0, row_len = 0, G = 1;
    size_t elt = 4;
    int64_t tile_bytes = 0, head_stride = 0, block_stride = 0, layer_stride = 0;
    float scale = 1.f;
    uint8_t *kv = nullptr;

    // host state
    std::vector<int32_t> table;   // [max_sessions][row_len]
    std::vector<uint8_t> is_open;
    std::vector<int64_t> len;
    std::vector<int32_t> n_assigned;
    BlockAllocator alloc;
    int64_t assigned = 0, reserved = 0;
    int32_t n_open = 0;

    // open plan
    bool plan_open = false;
    void *plan_stream = nullptr;
    int32_t n_seq = 0, T = 0, max_ntok = 0;
    bool all_single = false;
    bool pf_one_pass = false;  // every sequence takes one chunk-prefill row pass
    std::vector<int32_t> seq_sid, seq_ntok, seq_first;
    std::vector<int64_t> seq_pos0;
    std::vector<int32_t> tok_sid, tok_pos, tok_row, tok_block, tok_off;
    std::vector<int32_t> upd_idx, upd_val;
    std::vector<int32_t> pf_items;  // prefill work records (kPfItem ints per row pass)
    std::vector<int32_t> run_tok0, run_len;  // append runs: consecutive slots of one block
    std::vector<uint8_t> layer_done;

    // device
    int32_t max_tok = 0;           // capacity of one plan in tokens
    int32_t *d_table = nullptr;
    int32_t *d_meta = nullptr;     // packed plan metadata
    float2 *d_rope = nullptr;      // [max_tok][D/2]
    double *d_inv_freq = nullptr;  // [D/2]
    float *d_part = nullptr;       // decode split partials
    float *d_scratch = nullptr;    // the static partials workspace (not owned)
    size_t scratch_floats = 0;
    uint8_t *d_zero = nullptr;     // kZeroPage bytes of zeros (DMA source of absent blocks)
    size_t part_floats = 0;
    int32_t *h_stage[kStages] = {};
    hipEvent_t stage_ev[kStages] = {};
    bool stage_used[kStages] = {};
    int stage_i = 0;
    PlanView view{};
    int32_t *d_pf_items = nullptr;
    int32_t *d_run_tok0 = nullptr, *d_run_len = nullptr;
    int32_t resident_units = 0;    // decode work units resident on the whole GPU
    int32_t n_cu = 0;              // compute units of the pool's device
    int32_t pf_rows_cfg = 0;       // chunk-prefill rows per pass: 0 = chosen per plan
    int32_t pf_rows = 0;           // ... of the open plan
    int32_t decode_kernel = 0;     // 0 automatic, 1 vector, 2 matrix (test / tuning hook)
    int32_t last_split = 0;        // key segments of the most recent decode launch

    // stream order between plans: the per-plan device buffers (metadata, RoPE
    // table, split partials) are reused by the next plan, so a plan on another
    // stream first waits for everything issued on the previous plan's stream
    hipEvent_t order_ev = nullptr;
    bool have_last_stream = false;
    void *last_stream = nullptr;

    // failure injection (test hook): the launch point with this index fails
    int64_t fail_at = -1;

    // timing
    bool timing = false;
    std::vector<EventPair> ev_open[4];
    std::vector<hipEvent_t> ev_spare;
    int64_t t_launch[4] = {};
    double t_ms[4] = {};

    std::string last_error;
};

namespace {

mtn_status fail(mtn_pool *p, mtn_status s, const char *msg) noexcept {
    if (p) {
        try {
            p->last_error = msg;
        } catch (...) {
            // the status still says what failed
        }
    }
    return s;
}

// No C++ exception crosses the C ABI: a host allocation that fails inside an
// entry point returns MTN_ERR_HOST_MEMORY.  The planner reserves its
// per-plan vectors at pool creation, so plan_begin allocates only during
// validation, before it changes any state.
template <class F>
mtn_status guarded(mtn_pool *p, F &&f) noexcept {
    try {
        return f();
    } catch (...) {
        return fail(p, MTN_ERR_HOST_MEMORY, "host allocation failed");
    }
}

mtn_status hip_fail(mtn_pool *p, hipError_t e, const char *where) noexcept {
    if (p) {
        try {
            p->last_error = std::string(where) + ": " + hipGetErrorString(e);
        } catch (...) {
        }
    }
    return MTN_ERR_DEVICE;
}

#define HIP_TRY(p, expr)                                            \
    do {                                                            \
        hipError_t e_ = (expr);                                     \
        if (e_ != hipSuccess) return hip_fail((p), e_, #expr);      \
    } while (0)

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Bytes of one (layer, block, kv head) region: K tile + V^T tile of 16 x D
// elements, or for fp8 the code tiles plus 32 exponent bytes, padded to 128.
int64_t kv_head_stride(const mtn_pool_config *c) {
    if (c->kv_dtype == MTN_FP8_E4M3) return fp8_head_stride(c->head_dim);
    return 2 * (int64_t)kBlock * c->head_dim * (c->kv_dtype == MTN_BF16 ? 2 : 4);
}

mtn_status validate(const mtn_pool_config *c) {
    if (!c) return MTN_ERR_INVALID_ARG;
    if (c->n_layers < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1) return MTN_ERR_INVALID_ARG;
    if (c->n_q_heads % c->n_kv_heads) return MTN_ERR_INVALID_ARG;
    if (c->n_q_heads / c->n_kv_heads > 8) return MTN_ERR_UNSUPPORTED;
    if (c->head_dim != 64 && c->head_dim != 128) return MTN_ERR_UNSUPPORTED;
    if (c->block_size != kBlock) return MTN_ERR_UNSUPPORTED;
    if (c->max_chunk < 1 || c->max_sessions < 1 || c->n_blocks < 1) return MTN_ERR_INVALID_ARG;
    if (c->window == MTN_WINDOW_UNBOUNDED) {
        if (c->max_len < 1) return MTN_ERR_INVALID_ARG;
    } else {
        if (c->window < 1 || c->n_sink < 0) return MTN_ERR_INVALID_ARG;
        if ((int64_t)c->window + c->max_chunk + c->n_sink > (int64_t)1 << 30)
            return MTN_ERR_INVALID_ARG;
    }
    if (c->kv_dtype == MTN_FP8_E4M3) {
        // E4M3 codes in the pool, bf16 queries / keys / values / outputs
        if (c->io_dtype != MTN_BF16 || c->head_dim != 128) return MTN_ERR_UNSUPPORTED;
    } else {
        if (c->kv_dtype != MTN_F32 && c->kv_dtype != MTN_BF16) return MTN_ERR_INVALID_ARG;
        if (c->io_dtype != c->kv_dtype) return MTN_ERR_UNSUPPORTED;
    }
    if (!(c->rope_theta > 1.0)) return MTN_ERR_INVALID_ARG;
    if (c->softmax_scale < 0.f || !std::isfinite(c->softmax_scale)) return MTN_ERR_INVALID_ARG;
    if ((int64_t)c->max_sessions * c->max_chunk > (int64_t)1 << 24) return MTN_ERR_INVALID_ARG;
    {
        // block-table entries are addressed with 32-bit indices (plan updates)
        const int64_t ring = c->window == MTN_WINDOW_UNBOUNDED
                                 ? ceil_div(c->max_len, kBlock)
                                 : ceil_div((int64_t)c->window + c->max_chunk - 1, kBlock) +
                                       ceil_div(c->n_sink, kBlock);
        if ((int64_t)c->max_sessions * ring >= ((int64_t)1 << 31)) return MTN_ERR_INVALID_ARG;
    }
    if (c->flags & ~MTN_POOL_HOST_ONLY) return MTN_ERR_INVALID_ARG;
    return MTN_OK;
}

// Logical (block index in the session row, offset) of absolute position p.
inline void logical_slot(const mtn_pool *P, int64_t p, int32_t *lb, int32_t *off) {
    if (p < P->S) {
        *lb = (int32_t)(p / kBlock);
        *off = (int32_t)(p % kBlock);
        return;
    }
    int64_t sigma = P->unbounded ? p : (p - P->S) % P->R;
    *lb = P->nsb + (int32_t)(sigma / kBlock);
    *off = (int32_t)(sigma % kBlock);
}

// Number of not-yet-assigned logical blocks session `sid` touches when
// growing from L to L + n tokens.
int64_t new_blocks_needed(const mtn_pool *P, int32_t sid, int64_t L, int64_t n,
                          std::vector<uint8_t> &seen) {
    const int32_t *row = &P->table[(size_t)sid * P->row_len];
    int64_t need = 0;
    std::vector<int32_t> touched;
    for (int64_t p = L; p < L + n; ++p) {
        int32_t lb, off;
        logical_slot(P, p, &lb, &off);
        if (row[lb] < 0 && !seen[lb]) {
            seen[lb] = 1;
            touched.push_back(lb);
            ++need;
        }
    }
    for (int32_t lb : touched) seen[lb] = 0;
    return need;
}

mtn_status timing_begin(mtn_pool *P, hipStream_t s, hipEvent_t *out) {
    *out = nullptr;
    if (!P->timing) return MTN_OK;
    hipEvent_t e;
    if (!P->ev_spare.empty()) {
        e = P->ev_spare.back();
        P->ev_spare.pop_back();
    } else {
        HIP_TRY(P, hipEventCreate(&e));
    }
    HIP_TRY(P, hipEventRecord(e, s));
    *out = e;
    return MTN_OK;
}

mtn_status timing_end(mtn_pool *P, int cls, hipEvent_t a, hipStream_t s) {
    if (!P->timing || !a) return MTN_OK;
    hipEvent_t e;
    if (!P->ev_spare.empty()) {
        e = P->ev_spare.back();
        P->ev_spare.pop_back();
    } else {
        HIP_TRY(P, hipEventCreate(&e));
    }
    HIP_TRY(P, hipEventRecord(e, s));
    P->ev_open[cls].push_back({a, e});
    return MTN_OK;
}

// Return the blocks of the open plan's assignments (table index, physical
// block) to the pool, newest first.  The bitmap allocator then holds exactly
// its pre-plan free set, so later assignments are those of a pool that never
// saw the plan.  The device copy of the table keeps the stale entries, as
// after a session close: no kernel reads a logical block before a plan that
// assigns it again has uploaded the new entry.
void undo_assignments(mtn_pool *P) noexcept {
    for (size_t i = P->upd_idx.size(); i-- > 0;) {
        const int32_t idx = P->upd_idx[i];
        const int32_t sid = idx / P->row_len;
        P->table[(size_t)idx] = -1;
        P->alloc.give(P->upd_val[i]);
        P->n_assigned[sid]--;
        P->assigned--;
    }
    P->upd_idx.clear();
    P->upd_val.clear();
    if (P->unbounded) P->reserved = P->assigned;
}

// Abandon the open plan (nothing is committed).  Device work already issued
// for it wrote only slots of positions at or past each session's length;
// within one plan (at most max_chunk tokens per session) such a slot held
// no position that a later query can see, and the next plan over those
// positions writes them again before any query reads them.
void plan_abort_impl(mtn_pool *P) noexcept {
    undo_assignments(P);
    P->plan_open = false;
    P->n_seq = 0;
    P->T = 0;
}

// A point where device work is launched; the injected failure (test hook)
// fires here.  Host-only pools pass through the same points without launching.
mtn_status launch_gate(mtn_pool *P) {
    if (P->fail_at >= 0) {
        if (P->fail_at == 0) {
            P->fail_at = -1;
            return fail(P, MTN_ERR_DEVICE, "injected failure");
        }
        P->fail_at--;
    }
    return MTN_OK;
}

// Internal plan begin.  rows == nullptr packs io rows in plan order.
mtn_status plan_begin(mtn_pool *P, int32_t n_seq, const int32_t *sids, const int32_t *n_tok,
                      const int32_t *rows, void *stream) {
    if (P->plan_open) return fail(P, MTN_ERR_BAD_STATE, "a plan is already open");
    if (n_seq < 1 || n_seq > P->cfg.max_sessions || !sids || !n_tok)
        return fail(P, MTN_ERR_INVALID_ARG, "bad sequence count or null array");
    // ---- validation: nothing changes before every check has passed
    std::vector<uint8_t> seen((size_t)P->cfg.max_sessions, 0);
    int64_t T = 0;
    for (int32_t i = 0; i < n_seq; ++i) {
        int32_t sid = sids[i];
        if (sid < 0 || sid >= P->cfg.max_sessions || !P->is_open[sid])
            return fail(P, MTN_ERR_BAD_SESSION, "session not open");
        if (seen[sid]) return fail(P, MTN_ERR_INVALID_ARG, "duplicate session in plan");
        seen[sid] = 1;
        if (n_tok[i] < 1) return fail(P, MTN_ERR_INVALID_ARG, "n_tok < 1");
        // an io row list names one row per sequence: one-token sequences only
        // (the chunk prefill takes consecutive rows from a sequence's first)
        if (rows && n_tok[i] != 1) return fail(P, MTN_ERR_INVALID_ARG, "row list with n_tok > 1");
        if (n_tok[i] > P->cfg.max_chunk)
            return fail(P, MTN_ERR_CHUNK_TOO_LARGE, "n_tok > max_chunk");
        if (P->unbounded && P->len[sid] + n_tok[i] > P->cfg.max_len)
            return fail(P, MTN_ERR_SESSION_FULL, "session would pass max_len");
        if (!P->unbounded && P->len[sid] + n_tok[i] > ((int64_t)1 << 31) - 1)
            return fail(P, MTN_ERR_SESSION_FULL, "position overflow");
        T += n_tok[i];
    }
    {
        std::vector<uint8_t> lbseen((size_t)P->row_len, 0);
        int64_t need = 0;
        for (int32_t i = 0; i < n_seq; ++i)
            need += new_blocks_needed(P, sids[i], P->len[sids[i]], n_tok[i], lbseen);
        if (need > P->alloc.n_free()) return fail(P, MTN_ERR_POOL_EXHAUSTED, "pool exhausted");
    }
    int32_t *stage = nullptr;
    if (!P->host_only) {
        // wait until the staging buffer we are about to overwrite was consumed
        int si = P->stage_i;
        if (P->stage_used[si]) HIP_TRY(P, hipEventSynchronize(P->stage_ev[si]));
        stage = P->h_stage[si];
        if (P->have_last_stream && stream != P->last_stream) {
            HIP_TRY(P, hipEventRecord(P->order_ev, (hipStream_t)P->last_stream));
            HIP_TRY(P, hipStreamWaitEvent((hipStream_t)stream, P->order_ev, 0));
        }
        P->have_last_stream = true;
        P->last_stream = stream;
    }
    // ---- assignment (lowest free first, plan order)
    P->n_seq = n_seq;
    P->T = (int32_t)T;
    P->seq_sid.assign(sids, sids + n_seq);
    P->seq_ntok.assign(n_tok, n_tok + n_seq);
    P->seq_first.resize(n_seq);
    P->seq_pos0.resize(n_seq);
    P->tok_sid.resize(T);
    P->tok_pos.resize(T);
    P->tok_row.resize(T);
    P->tok_block.resize(T);
    P->tok_off.resize(T);
    P->upd_idx.clear();
    P->upd_val.clear();
    P->max_ntok = 0;
    int32_t t = 0;
    for (int32_t i = 0; i < n_seq; ++i) {
        int32_t sid = sids[i];
        int32_t *row = &P->table[(size_t)sid * P->row_len];
        P->seq_first[i] = t;
        P->seq_pos0[i] = P->len[sid];
        P->max_ntok = std::max(P->max_ntok, n_tok[i]);
        for (int32_t j = 0; j < n_tok[i]; ++j, ++t) {
            int64_t pos = P->len[sid] + j;
            int32_t lb, off;
            logical_slot(P, pos, &lb, &off);
            if (row[lb] < 0) {
                int64_t b = P->alloc.take();
                row[lb] = (int32_t)b;
                P->n_assigned[sid]++;
                P->assigned++;
                P->upd_idx.push_back(sid * P->row_len + lb);
                P->upd_val.push_back((int32_t)b);
            }
            P->tok_sid[t] = sid;
            P->tok_pos[t] = (int32_t)pos;
            P->tok_row[t] = rows ? rows[i] : t;
            P->tok_block[t] = row[lb];
            P->tok_off[t] = off;
        }
    }
    if (P->unbounded) P->reserved = P->assigned;
    P->all_single = (P->max_ntok == 1);
    // append runs: maximal stretches of one sequence's tokens in consecutive
    // slots of one block (the append kernel writes each with one wave per kv
    // head, K rows and V^T row segments contiguous)
    P->run_tok0.clear();
    P->run_len.clear();
    for (int32_t i = 0, tt = 0; i < n_seq; ++i)
        for (int32_t j = 0; j < n_tok[i]; ++j, ++tt) {
            const bool cont = j > 0 && P->tok_block[tt] == P->tok_block[tt - 1] &&
                              P->tok_off[tt] == P->tok_off[tt - 1] + 1;
            if (cont) {
                P->run_len.back()++;
            } else {
                P->run_tok0.push_back(tt);
                P->run_len.push_back(1);
            }
        }
    P->pf_items.clear();
    {
        // Rows per prefill pass.  Few sequences leave most CUs idle with full
        // passes (one workgroup per sequence and kv head); then 128-row passes
        // give each sequence more workgroups (each reading the keys its rows
        // see), and a pass whose waves hold one tile skips the empty second.
        int64_t rpp = P->pf_rows_cfg ? P->pf_rows_cfg : prefill_rows_per_pass();
        if (!P->pf_rows_cfg && P->n_cu > 0) {
            int64_t wgs = 0;
            for (int32_t i = 0; i < n_seq; ++i) wgs += ceil_div((int64_t)n_tok[i] * P->G, rpp);
            if (2 * wgs * P->cfg.n_kv_heads <= P->n_cu && prefill_pass_rows_valid(128)) rpp = 128;
        }
        P->pf_rows = (int32_t)rpp;
        // one record per (sequence, row pass) with everything its workgroup
        // needs before the first copy, so that it takes one metadata load.
        // The prefill takes io row (row of t0) + j for token t0 + j: plans
        // with an explicit row list (frame_step's decode rounds) carry one
        // token per sequence and never reach it.
        for (int32_t i = 0; i < n_seq; ++i) {
            const int32_t t0 = P->seq_first[i];
            for (int64_t p = 0; p * rpp < (int64_t)n_tok[i] * P->G; ++p) {
                const int32_t rec[kPfItem] = {(int32_t)p, t0, n_tok[i], sids[i],
                                              (int32_t)P->seq_pos0[i], P->tok_row[t0], 0, 0};
                P->pf_items.insert(P->pf_items.end(), rec, rec + kPfItem);
            }
        }
        P->pf_one_pass = P->pf_items.size() == (size_t)kPfItem * n_seq;
    }
    P->layer_done.assign((size_t)P->cfg.n_layers, 0);
    P->plan_open = true;
    P->plan_stream = stream;
    if (P->host_only) return MTN_OK;

    // ---- upload: one packed blob, then the apply kernel (table + RoPE)
    const int32_t U = (int32_t)P->upd_idx.size();
    int32_t *h = stage;
    size_t o = 0;
    auto put = [&](const int32_t *src, int32_t n) {
        std::memcpy(h + o, src, sizeof(int32_t) * (size_t)n);
        o += (size_t)n;
    };
    put(P->tok_sid.data(), T);
    put(P->tok_pos.data(), T);
    put(P->tok_row.data(), T);
    put(P->tok_block.data(), T);
    put(P->tok_off.data(), T);
    put(P->upd_idx.data(), U);
    put(P->upd_val.data(), U);
    const size_t o_items = (o + kPfItem - 1) / kPfItem * kPfItem;  // records 32-byte aligned
    while (o < o_items) h[o++] = 0;
    put(P->pf_items.data(), (int32_t)P->pf_items.size());
    const int32_t NR = (int32_t)P->run_tok0.size();
    put(P->run_tok0.data(), NR);
    put(P->run_len.data(), NR);
    hipStream_t s = (hipStream_t)stream;
    int32_t *d = P->d_meta;
    // a failed upload abandons the plan: the pool is as before the call
    auto upload_fail = [&](hipError_t e, const char *where) {
        plan_abort_impl(P);
        return hip_fail(P, e, where);
    };
    hipError_t he = hipMemcpyAsync(d, h, o * sizeof(int32_t), hipMemcpyHostToDevice, s);
    if (he != hipSuccess) return upload_fail(he, "plan upload");
    he = hipEventRecord(P->stage_ev[P->stage_i], s);
    if (he != hipSuccess) return upload_fail(he, "plan upload event");
    P->stage_used[P->stage_i] = true;
    P->stage_i = (P->stage_i + 1) % kStages;
    P->view.tok_sid = d;
    P->view.tok_pos = d + T;
    P->view.tok_row = d + 2 * T;
    P->view.tok_block = d + 3 * T;
    P->view.tok_off = d + 4 * T;
    P->view.rope = P->d_rope;
    P->view.n_tok = (int32_t)T;
    const int32_t *d_upd_idx = d + 5 * T;
    P->d_pf_items = d + o_items;
    P->d_run_tok0 = P->d_pf_items + P->pf_items.size();
    P->d_run_len = P->d_run_tok0 + NR;
    he = launch_plan_apply(d_upd_idx, d_upd_idx + U, U, P->d_table, P->view.tok_pos, (int32_t)T,
                           P->d_inv_freq, P->cfg.head_dim / 2, P->d_rope, s);
    if (he != hipSuccess) return upload_fail(he, "launch_plan_apply");
    return MTN_OK;
}

mtn_status plan_commit(mtn_pool *P) {
    if (!P->plan_open) return fail(P, MTN_ERR_BAD_STATE, "no open plan");
    if (!P->host_only)
        for (auto d : P->layer_done)
            if (!d) return fail(P, MTN_ERR_BAD_STATE, "commit before every layer was appended");
    for (int32_t i = 0; i < P->n_seq; ++i) P->len[P->seq_sid[i]] += P->seq_ntok[i];
    P->plan_open = false;
    return MTN_OK;
}

PoolGeom geom(const mtn_pool *P) {
    PoolGeom g;
    g.kv = P->kv;
    g.layer_stride = P->layer_stride;
    g.block_stride = P->block_stride;
    g.head_stride = P->head_stride;
    g.tile_bytes = P->tile_bytes;
    g.table = P->d_table;
    g.row_len = P->row_len;
    g.n_sink = P->S;
    g.window = P->W;
    g.ring = P->R;
    g.n_sink_blocks = P->nsb;
    g.hq = P->cfg.n_q_heads;
    g.hkv = P->cfg.n_kv_heads;
    g.d = P->cfg.head_dim;
    return g;
}

mtn_status check_call(mtn_pool *P, int32_t layer, void *stream) {
    if (!P) return MTN_ERR_INVALID_ARG;
    if (P->host_only) return fail(P, MTN_ERR_BAD_STATE, "host-only pool has no device path");
    if (!P->plan_open) return fail(P, MTN_ERR_BAD_STATE, "no open plan");
    if (stream != P->plan_stream) return fail(P, MTN_ERR_INVALID_ARG, "stream differs from plan's");
    if (layer < 0 || layer >= P->cfg.n_layers) return fail(P, MTN_ERR_INVALID_ARG, "bad layer");
    return MTN_OK;
}

mtn_status append_impl(mtn_pool *P, int32_t layer, const void *k, const void *v, void *stream) {
    mtn_status st = launch_gate(P);
    if (st) return st;
    if (P->host_only) {  // frame_step on a host-only pool: planning only
        P->layer_done[layer] = 1;
        return MTN_OK;
    }
    hipStream_t s = (hipStream_t)stream;
    hipEvent_t e0;
    st = timing_begin(P, s, &e0);
    if (st) return st;
    if (P->cfg.kv_dtype == MTN_FP8_E4M3)
        HIP_TRY(P, launch_append_fp8(geom(P), P->view, layer, k, v, s));
    else
        HIP_TRY(P, launch_append(P->cfg.kv_dtype, geom(P), P->view, layer, k, v, P->d_run_tok0,
                                 P->d_run_len, (int32_t)P->run_tok0.size(), s));
    st = timing_end(P, 0, e0, s);
    if (st) return st;
    P->layer_done[layer] = 1;
    return MTN_OK;
}

AttnArgs attn_args(mtn_pool *P, int32_t layer, const void *q, void *out, float *lse,
                   int32_t n_split) {
    AttnArgs a;
    a.g = geom(P);
    a.p = P->view;
    a.layer = layer;
    a.q = q;
    a.out = out;
    a.lse = lse;
    a.part = P->d_part;
    a.n_split = n_split;
    a.scale_log2 = P->scale * 1.4426950408889634f;
    a.zero_page = P->d_zero;
    a.k_new = nullptr;
    a.v_new = nullptr;
    return a;
}

// bf16 decode kernel: the MFMA kernel (per-wave LDS rings, all heads of a KV
// group per block on matrix cores) for D = 128 and G = 8, the vector kernel
// otherwise.  Measured: at the 128-session G = 8 shape 6.63 TB/s against 5.84
// for the vector kernel; at the 64-session G = 1 and 256-session G = 4 shapes
// the vector kernel's one-wave workgroups win (6.86 and 6.68 TB/s against
// 6.61 and 6.53).
// mtn_pool_set_decode_kernel can force either kernel where it exists.
bool use_mfma_bf16(const mtn_pool *P) {
    if (P->cfg.kv_dtype != MTN_BF16 || !attn_mfma_bf16_supported(P->cfg.head_dim, P->G))
        return false;
    if (P->decode_kernel == 1) return false;
    if (P->decode_kernel == 2) return true;
    return P->G == 8;
}

// decode work units the split rule counts as one round on the whole GPU: the
// kernels' own per-CU figure (the vector decode's occupancy; for the
// matrix-core decode the workgroups holding about 64 KiB of copies in flight)
int32_t count_resident_units(const mtn_pool *P) {
    const mtn_pool_config &c = P->cfg;
    const int per_cu = c.kv_dtype == MTN_FP8_E4M3 ? attn_fp8_resident_per_cu(P->G)
                       : use_mfma_bf16(P)         ? attn_mfma_bf16_resident_per_cu(P->G)
                                                  : attn_valu_resident_per_cu(c.kv_dtype, c.head_dim, P->G);
    return P->n_cu * per_cu;
}

// Decode split heuristic.  A unit (query, kv head, segment) streams its keys
// through an LDS ring whose pipeline fills at the start and drains at the
// end, so units should be long, and a partly filled last round of units
// leaves CUs idle.  So: if the unsplit units already fill the resident slots,
// keep them whole; otherwise split just enough to fill one round, keeping at
// least 16 blocks per segment.
int32_t auto_split(const mtn_pool *P, int32_t n_items) {
    int64_t units = (int64_t)n_items * P->cfg.n_kv_heads;
    int64_t max_keys = P->unbounded ? P->cfg.max_len : (int64_t)P->S + P->W;
    int64_t blocks = ceil_div(max_keys, kBlock) + 1;
    int64_t resident = std::max<int32_t>(P->resident_units, 1);
    if (units >= resident) return 1;
    int64_t sp = resident / std::max<int64_t>(units, 1);
    sp = std::min<int64_t>(sp, std::max<int64_t>(1, blocks / 16));
    return (int32_t)std::max<int64_t>(1, std::min<int64_t>(sp, kMaxSplit));
}

// k_new / v_new non-null: the decode also appends the planned tokens of this
// layer (each is the newest key of its own query), in the same launch.
// The split partials workspace holds kMaxSplit segments of every query a
// plan can carry (max_sessions), so every split 1 <= n_split <= kMaxSplit runs
// as asked.
// part / part_floats: another partials workspace (the static one); such a
// call records no timing events.
mtn_status decode_impl(mtn_pool *P, int32_t layer, const void *q, void *out, float *lse,
                       int32_t n_split, void *stream, const void *k_new = nullptr,
                       const void *v_new = nullptr, float *part = nullptr,
                       size_t part_floats = 0) {
    mtn_status st = launch_gate(P);
    if (st) return st;
    if (P->host_only) {  // frame_step on a host-only pool: planning only
        if (k_new) P->layer_done[layer] = 1;
        return MTN_OK;
    }
    hipStream_t s = (hipStream_t)stream;
    if (n_split == 0) n_split = auto_split(P, P->T);
    const bool events = part == nullptr;
    if (!part) {
        part = P->d_part;
        part_floats = P->part_floats;
    }
    if (n_split > 1 &&
        (size_t)P->T * P->cfg.n_q_heads * n_split * (P->cfg.head_dim + 2) > part_floats)
        return fail(P, MTN_ERR_INVALID_ARG, "split partials exceed the workspace");
    AttnArgs a = attn_args(P, layer, q, out, lse, n_split);
    a.part = part;
    a.k_new = k_new;
    a.v_new = v_new;
    hipEvent_t e0 = nullptr;
    if (events) {
        st = timing_begin(P, s, &e0);
        if (st) return st;
    }
    if (P->cfg.kv_dtype == MTN_FP8_E4M3)
        HIP_TRY(P, launch_attn_fp8(a, s));
    else if (use_mfma_bf16(P))
        HIP_TRY(P, launch_attn_mfma_bf16(a, s));
    else
        HIP_TRY(P, launch_attn_valu(P->cfg.kv_dtype, a, s));
    if (events) {
        st = timing_end(P, 2, e0, s);
        if (st) return st;
    }
    P->last_split = n_split;
    if (k_new) P->layer_done[layer] = 1;
    if (n_split > 1) {
        if (events) {
            st = timing_begin(P, s, &e0);
            if (st) return st;
        }
        HIP_TRY(P, launch_merge(P->cfg.io_dtype, a, s));  // writes io rows
        if (events) {
            st = timing_end(P, 3, e0, s);
            if (st) return st;
        }
    }
    return MTN_OK;
}

// Whether frame_step fuses the chunk append into the chunk prefill: the fp8
// pool's matrix-core prefill with every sequence in one row pass (its
// workgroup is then the only reader of the sequence's blocks of its kv head),
// and at most two workgroups per CU.  Each workgroup pays the append's work
// before its first stage: measured, that costs less than the quantizing
// append launch at two rounds of workgroups per CU (128 sessions x 4 kv
// heads), more at eight (256 sessions x 8 kv heads), and for the bf16 pool
// no less than its append launch.
bool prefill_fuses_append(const mtn_pool *P) {
    const int64_t wgs = (int64_t)(P->pf_items.size() / kPfItem) * P->cfg.n_kv_heads;
    return !P->all_single && P->pf_one_pass && P->n_cu > 0 && wgs <= 2 * (int64_t)P->n_cu &&
           P->cfg.kv_dtype == MTN_FP8_E4M3 &&
           prefill_mfma_supported(P->cfg.kv_dtype, P->cfg.head_dim, P->G);
}

// k_new / v_new non-null (only when prefill_fuses_append): the launch also
// appends the planned tokens, and the layer counts as appended.
mtn_status prefill_impl(mtn_pool *P, int32_t layer, const void *q, void *out, float *lse,
                        void *stream, const void *k_new = nullptr, const void *v_new = nullptr) {
    hipStream_t s = (hipStream_t)stream;
    if (P->all_single) return decode_impl(P, layer, q, out, lse, 0, stream);
    mtn_status st = launch_gate(P);
    if (st) return st;
    if (P->host_only) {
        if (k_new) P->layer_done[layer] = 1;
        return MTN_OK;
    }
    AttnArgs a = attn_args(P, layer, q, out, lse, 1);
    a.k_new = k_new;
    a.v_new = v_new;
    hipEvent_t e0;
    st = timing_begin(P, s, &e0);
    if (st) return st;
    if (prefill_mfma_supported(P->cfg.kv_dtype, P->cfg.head_dim, P->G)) {
        HIP_TRY(P, launch_prefill_mfma(P->cfg.kv_dtype, a, P->d_pf_items,
                                       (int32_t)(P->pf_items.size() / kPfItem), P->pf_rows, P->d_zero, s));
    } else {
        HIP_TRY(P, launch_attn_valu(P->cfg.kv_dtype, a, s));
    }
    st = timing_end(P, 1, e0, s);
    if (st) return st;
    if (k_new) P->layer_done[layer] = 1;
    return MTN_OK;
}

// The plans of one frame (after mtn_frame_step's validation): the chunk plan
// with every layer's append + chunk prefill (or the fused one-token decode),
// then one plan per decode round.  Returns at the first error, with the
// failing plan still open.
mtn_status frame_plans(mtn_pool *P, const mtn_frame_batch *b, void *stream, int64_t Tc,
                       int32_t max_dec, std::vector<int32_t> &sids, std::vector<int32_t> &ones,
                       std::vector<int32_t> &rows) {
    const int32_t n = b->n_seq, L = P->cfg.n_layers;
    const int32_t Hq = P->cfg.n_q_heads, Hkv = P->cfg.n_kv_heads;
    const size_t e = P->elt, D = (size_t)P->cfg.head_dim;
    // host-only pools take null buffers: no offset is formed from them
    auto off = [&](const void *base, size_t elems) -> const void * {
        return base ? (const void *)((const uint8_t *)base + elems * e) : nullptr;
    };
    mtn_status st = plan_begin(P, n, b->sids, b->chunk_len, nullptr, stream);
    if (st) return st;
    for (int32_t l = 0; l < L; ++l) {
        const size_t rq = (size_t)l * Tc * Hq * D, rk = (size_t)l * Tc * Hkv * D;
        float *lse = b->lse_chunk ? b->lse_chunk + (size_t)l * Tc * Hq : nullptr;
        if (P->all_single) {  // one-token chunks: decode with the append fused in
            st = decode_impl(P, l, off(b->q_chunk, rq), (void *)off(b->out_chunk, rq), lse,
                             b->n_split, stream, off(b->k_chunk, rk), off(b->v_chunk, rk));
        } else if (prefill_fuses_append(P)) {  // append fused into the prefill
            st = prefill_impl(P, l, off(b->q_chunk, rq), (void *)off(b->out_chunk, rq), lse,
                              stream, off(b->k_chunk, rk), off(b->v_chunk, rk));
        } else {
            st = append_impl(P, l, off(b->k_chunk, rk), off(b->v_chunk, rk), stream);
            if (st) return st;
            st = prefill_impl(P, l, off(b->q_chunk, rq), (void *)off(b->out_chunk, rq), lse,
                              stream);
        }
        if (st) return st;
    }
    st = plan_commit(P);
    if (st) return st;
    for (int32_t j = 0; j < max_dec; ++j) {
        sids.clear();
        rows.clear();
        for (int32_t i = 0; i < n; ++i)
            if (b->n_decode[i] > j) {
                sids.push_back(b->sids[i]);
                rows.push_back(i);
            }
        ones.assign(sids.size(), 1);
        st = plan_begin(P, (int32_t)sids.size(), sids.data(), ones.data(), rows.data(), stream);
        if (st) return st;
        for (int32_t l = 0; l < L; ++l) {
            const size_t base = ((size_t)j * L + l) * n;
            float *lse = b->lse_dec ? b->lse_dec + base * Hq : nullptr;
            st = decode_impl(P, l, off(b->q_dec, base * Hq * D),
                             (void *)off(b->out_dec, base * Hq * D), lse, b->n_split, stream,
                             off(b->k_dec, base * Hkv * D), off(b->v_dec, base * Hkv * D));
            if (st) return st;
        }
        st = plan_commit(P);
        if (st) return st;
    }
    return MTN_OK;
}

mtn_status pool_init(mtn_pool *P, const mtn_pool_config *cfg, void *kv_dev, void *stream);

}  // namespace

extern "C" {

const char *mtn_status_string(mtn_status s) {
    switch (s) {
        case MTN_OK: return "ok";
        case MTN_ERR_INVALID_ARG: return "invalid argument";
        case MTN_ERR_BAD_SESSION: return "bad session id";
        case MTN_ERR_CHUNK_TOO_LARGE: return "chunk larger than max_chunk";
        case MTN_ERR_NO_SESSION_SLOT: return "no free session slot";
        case MTN_ERR_POOL_EXHAUSTED: return "KV pool exhausted";
        case MTN_ERR_SESSION_FULL: return "session at max_len";
        case MTN_ERR_DEVICE: return "device error";
        case MTN_ERR_BAD_STATE: return "call out of order";
        case MTN_ERR_UNSUPPORTED: return "unsupported shape or dtype";
        case MTN_ERR_HOST_MEMORY: return "host allocation failed";
        default: return "unknown status";
    }
}

const char *mtn_pool_last_error(const mtn_pool *pool) {
    return pool ? pool->last_error.c_str() : "";
}

mtn_status mtn_pool_required_bytes(const mtn_pool_config *cfg, size_t *kv_bytes) {
    mtn_status st = validate(cfg);
    if (st) return st;
    if (!kv_bytes) return MTN_ERR_INVALID_ARG;
    size_t per_block = (size_t)cfg->n_kv_heads * (size_t)kv_head_stride(cfg);
    *kv_bytes = per_block * (size_t)cfg->n_blocks * (size_t)cfg->n_layers;
    return MTN_OK;
}

mtn_status mtn_pool_create(const mtn_pool_config *cfg, void *kv_dev, size_t kv_bytes,
                           void *stream, mtn_pool **out) {
    if (!out) return MTN_ERR_INVALID_ARG;
    size_t need;
    mtn_status st = mtn_pool_required_bytes(cfg, &need);
    if (st) return st;
    bool host_only = cfg->flags & MTN_POOL_HOST_ONLY;
    if (!host_only) {
        if (!kv_dev || kv_bytes < need || ((uintptr_t)kv_dev & 255)) return MTN_ERR_INVALID_ARG;
        const int g = cfg->n_q_heads / cfg->n_kv_heads;
        if (cfg->kv_dtype == MTN_FP8_E4M3 ? !attn_fp8_supported(cfg->head_dim, g)
                                          : !attn_valu_supported(cfg->kv_dtype, cfg->head_dim, g))
            return MTN_ERR_UNSUPPORTED;
    }
    mtn_pool *P = new (std::nothrow) mtn_pool();
    if (!P) return MTN_ERR_HOST_MEMORY;
    try {
        st = pool_init(P, cfg, kv_dev, stream);
    } catch (...) {
        st = MTN_ERR_HOST_MEMORY;
    }
    if (st) {
        mtn_pool_destroy(P);
        return st;
    }
    *out = P;
    return MTN_OK;
}

}  // extern "C"

namespace {

// Everything of pool creation past validation; on failure the caller
// destroys the partly built pool.
mtn_status pool_init(mtn_pool *P, const mtn_pool_config *cfg, void *kv_dev, void *stream) {
    const bool host_only = cfg->flags & MTN_POOL_HOST_ONLY;
    P->cfg = *cfg;
    P->host_only = host_only;
    P->unbounded = cfg->window == MTN_WINDOW_UNBOUNDED;
    P->G = cfg->n_q_heads / cfg->n_kv_heads;
    P->elt = cfg->io_dtype == MTN_BF16 ? 2 : 4;  // io element size
    if (P->unbounded) {
        P->S = 0;
        P->W = -1;
        P->nsb = 0;
        P->R = (int32_t)(ceil_div(cfg->max_len, kBlock) * kBlock);
    } else {
        P->S = cfg->n_sink;
        P->W = cfg->window;
        P->nsb = (int32_t)ceil_div(cfg->n_sink, kBlock);
        P->R = (int32_t)(ceil_div((int64_t)cfg->window + cfg->max_chunk - 1, kBlock) * kBlock);
    }
    P->row_len = P->nsb + P->R / kBlock;
    P->tile_bytes = (int64_t)kBlock * cfg->head_dim * (cfg->kv_dtype == MTN_FP8_E4M3 ? 1 : (int64_t)P->elt);
    P->head_stride = kv_head_stride(cfg);
    P->block_stride = P->head_stride * cfg->n_kv_heads;
    P->layer_stride = P->block_stride * cfg->n_blocks;
    P->scale = cfg->softmax_scale > 0.f ? cfg->softmax_scale
                                        : (float)(1.0 / std::sqrt((double)cfg->head_dim));
    P->kv = (uint8_t *)kv_dev;
    P->table.assign((size_t)cfg->max_sessions * P->row_len, -1);
    P->is_open.assign((size_t)cfg->max_sessions, 0);
    P->len.assign((size_t)cfg->max_sessions, 0);
    P->n_assigned.assign((size_t)cfg->max_sessions, 0);
    P->alloc.reset(cfg->n_blocks);
    P->max_tok = cfg->max_sessions * cfg->max_chunk;
    // the planner's per-plan vectors at their largest, so that planning
    // allocates nothing once validation has passed
    P->seq_sid.reserve((size_t)cfg->max_sessions);
    P->seq_ntok.reserve((size_t)cfg->max_sessions);
    P->seq_first.reserve((size_t)cfg->max_sessions);
    P->seq_pos0.reserve((size_t)cfg->max_sessions);
    for (auto *v : {&P->tok_sid, &P->tok_pos, &P->tok_row, &P->tok_block, &P->tok_off, &P->upd_idx,
                    &P->upd_val, &P->run_tok0, &P->run_len})
        v->reserve((size_t)P->max_tok);
    P->pf_items.reserve(kPfItem * ((size_t)P->max_tok * P->G / 128 + (size_t)cfg->max_sessions + 1));
    P->layer_done.reserve((size_t)cfg->n_layers);
    if (!host_only) {
        auto bail = [&](hipError_t e, const char *w) {
            (void)e;
            (void)w;
            return MTN_ERR_DEVICE;
        };
        hipError_t e;
        size_t tbl = sizeof(int32_t) * P->table.size();
        if ((e = hipMalloc(&P->d_table, tbl)) != hipSuccess) return bail(e, "table");
        if ((e = hipMemcpyAsync(P->d_table, P->table.data(), tbl, hipMemcpyHostToDevice,
                                (hipStream_t)stream)) != hipSuccess)
            return bail(e, "table upload");
        // per plan: 5 T token fields, 2 U table updates (U <= T), kPfItem per
        // prefill pass (<= T G / 128 + n_seq passes, aligned to a record) and 2
        // per append run (<= T)
        size_t meta = sizeof(int32_t) * ((size_t)P->max_tok * 9 +
                                         kPfItem * ((size_t)P->max_tok * P->G / 128 +
                                                    (size_t)cfg->max_sessions + 1) +
                                         64);
        if ((e = hipMalloc(&P->d_meta, meta)) != hipSuccess) return bail(e, "meta");
        for (int i = 0; i < kStages; ++i) {
            if ((e = hipHostMalloc(&P->h_stage[i], meta, hipHostMallocDefault)) != hipSuccess)
                return bail(e, "stage");
            if ((e = hipEventCreateWithFlags(&P->stage_ev[i], hipEventDisableTiming)) != hipSuccess)
                return bail(e, "event");
        }
        size_t half = (size_t)cfg->head_dim / 2;
        if ((e = hipMalloc(&P->d_rope, sizeof(float2) * half * (size_t)P->max_tok)) != hipSuccess)
            return bail(e, "rope");
        std::vector<double> inv(half);
        for (size_t i = 0; i < half; ++i)
            inv[i] = std::pow(cfg->rope_theta, -2.0 * (double)i / (double)cfg->head_dim);
        if ((e = hipMalloc(&P->d_inv_freq, sizeof(double) * half)) != hipSuccess)
            return bail(e, "inv_freq");
        if ((e = hipMemcpy(P->d_inv_freq, inv.data(), sizeof(double) * half,
                           hipMemcpyHostToDevice)) != hipSuccess)
            return bail(e, "inv_freq upload");
        // zero page: at least one whole (block, head) pair, K + V^T, at the
        // largest element size and head dim
        if ((e = hipMalloc(&P->d_zero, kZeroPage)) != hipSuccess) return bail(e, "zero page");
        if ((e = hipMemsetAsync(P->d_zero, 0, kZeroPage, (hipStream_t)stream)) != hipSuccess)
            return bail(e, "zero page clear");
        P->part_floats = (size_t)cfg->max_sessions * cfg->n_q_heads * kMaxSplit * (cfg->head_dim + 2);
        if ((e = hipMalloc(&P->d_part, sizeof(float) * P->part_floats)) != hipSuccess)
            return bail(e, "partials");
        if ((e = scratch_buffer(&P->d_scratch, &P->scratch_floats)) != hipSuccess)
            return bail(e, "static scratch address");
        int dev = 0, n_cu = 0;
        if ((e = hipGetDevice(&dev)) != hipSuccess) return bail(e, "device");
        if ((e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev)) !=
            hipSuccess)
            return bail(e, "cu count");
        P->n_cu = n_cu;
        P->resident_units = count_resident_units(P);
        if ((e = hipEventCreateWithFlags(&P->order_ev, hipEventDisableTiming)) != hipSuccess)
            return bail(e, "event");
        if ((e = hipStreamSynchronize((hipStream_t)stream)) != hipSuccess)
            return bail(e, "sync");
    }
    return MTN_OK;
}

}  // namespace

extern "C" {

void mtn_pool_destroy(mtn_pool *P) {
    if (!P) return;
    if (!P->host_only) {
        (void)hipDeviceSynchronize();
        (void)hipFree(P->d_table);
        (void)hipFree(P->d_meta);
        (void)hipFree(P->d_rope);
        (void)hipFree(P->d_inv_freq);
        (void)hipFree(P->d_part);
        (void)hipFree(P->d_zero);
        for (int i = 0; i < kStages; ++i) {
            if (P->h_stage[i]) (void)hipHostFree(P->h_stage[i]);
            if (P->stage_ev[i]) (void)hipEventDestroy(P->stage_ev[i]);
        }
        for (auto &v : P->ev_open)
            for (auto &pr : v) {
                (void)hipEventDestroy(pr.a);
                (void)hipEventDestroy(pr.b);
            }
        for (auto e : P->ev_spare) (void)hipEventDestroy(e);
        if (P->order_ev) (void)hipEventDestroy(P->order_ev);
    }
    delete P;
}

mtn_status mtn_session_open(mtn_pool *P, int32_t *sid_out) {
    return guarded(P, [&]() -> mtn_status {
        if (!P || !sid_out) return MTN_ERR_INVALID_ARG;
        int32_t sid = -1;
        for (int32_t i = 0; i < P->cfg.max_sessions; ++i)
            if (!P->is_open[i]) {
                sid = i;
                break;
            }
        if (sid < 0) return fail(P, MTN_ERR_NO_SESSION_SLOT, "no free session slot");
        if (!P->unbounded) {
            if (P->reserved + P->row_len > P->cfg.n_blocks)
                return fail(P, MTN_ERR_POOL_EXHAUSTED, "reservation exceeds pool capacity");
            P->reserved += P->row_len;
        }
        P->is_open[sid] = 1;
        P->len[sid] = 0;
        P->n_assigned[sid] = 0;
        P->n_open++;
        *sid_out = sid;
        return MTN_OK;
    });
}

mtn_status mtn_session_close(mtn_pool *P, int32_t sid) {
    return guarded(P, [&]() -> mtn_status {
        if (!P) return MTN_ERR_INVALID_ARG;
        if (P->plan_open) return fail(P, MTN_ERR_BAD_STATE, "plan open");
        if (sid < 0 || sid >= P->cfg.max_sessions || !P->is_open[sid])
            return fail(P, MTN_ERR_BAD_SESSION, "session not open");
        int32_t *row = &P->table[(size_t)sid * P->row_len];
        for (int32_t j = 0; j < P->row_len; ++j) {
            if (row[j] >= 0) {
                P->alloc.give(row[j]);
                P->assigned--;
                row[j] = -1;
            }
        }
        if (!P->unbounded) P->reserved -= P->row_len;
        else P->reserved = P->assigned;
        P->is_open[sid] = 0;
        P->len[sid] = 0;
        P->n_assigned[sid] = 0;
        P->n_open--;
        // The device copy of the row is left as is: kernels still in flight may
        // read it, and a reopened session only ever reads logical blocks that its
        // own plans assigned (and uploaded, in stream order) again.
        return MTN_OK;
    });
}

mtn_status mtn_plan_begin(mtn_pool *P, int32_t n_seq, const int32_t *sids, const int32_t *n_tok,
                          void *stream) {
    return guarded(P, [&]() -> mtn_status {
        if (!P) return MTN_ERR_INVALID_ARG;
        return plan_begin(P, n_seq, sids, n_tok, nullptr, stream);
    });
}

mtn_status mtn_plan_commit(mtn_pool *P) {
    return guarded(P, [&]() -> mtn_status {
        if (!P) return MTN_ERR_INVALID_ARG;
        return plan_commit(P);
    });
}

mtn_status mtn_plan_abort(mtn_pool *P) {
    return guarded(P, [&]() -> mtn_status {
        if (!P) return MTN_ERR_INVALID_ARG;
        if (!P->plan_open) return fail(P, MTN_ERR_BAD_STATE, "no open plan");
        plan_abort_impl(P);
        return MTN_OK;
    });
}

// Activation buffers (q, k, v, out) are read and written in 16-byte vectors.
static bool bad_buf(const void *p) { return !p || ((uintptr_t)p & 15); }

mtn_status mtn_frame_append_kv(mtn_pool *P, int32_t layer, const void *k, const void *v,
                               void *stream) {
    return guarded(P, [&]() -> mtn_status {
        mtn_status st = check_call(P, layer, stream);
        if (st) return st;
        if (bad_buf(k) || bad_buf(v)) return fail(P, MTN_ERR_INVALID_ARG, "null or misaligned k or v");
        return append_impl(P, layer, k, v, stream);
    });
}

mtn_status mtn_attend_chunk_prefill(mtn_pool *P, int32_t layer, const void *q, void *out,
                                    float *lse, void *stream) {
    return guarded(P, [&]() -> mtn_status {
        mtn_status st = check_call(P, layer, stream);
        if (st) return st;
        if (bad_buf(q) || bad_buf(out)) return fail(P, MTN_ERR_INVALID_ARG, "null or misaligned q or out");
        if (!P->layer_done[layer]) return fail(P, MTN_ERR_BAD_STATE, "layer not appended");
        return prefill_impl(P, layer, q, out, lse, stream);
    });
}

mtn_status mtn_attend_decode(mtn_pool *P, int32_t layer, const void *q, void *out, float *lse,
                             int32_t n_split, void *stream) {
    return guarded(P, [&]() -> mtn_status {
        mtn_status st = check_call(P, layer, stream);
        if (st) return st;
        if (bad_buf(q) || bad_buf(out)) return fail(P, MTN_ERR_INVALID_ARG, "null or misaligned q or out");
        if (!P->all_single) return fail(P, MTN_ERR_BAD_STATE, "decode needs n_tok == 1 everywhere");
        if (n_split < 0 || n_split > kMaxSplit) return fail(P, MTN_ERR_INVALID_ARG, "bad n_split");
        if (!P->layer_done[layer]) return fail(P, MTN_ERR_BAD_STATE, "layer not appended");
        return decode_impl(P, layer, q, out, lse, n_split, stream);
    });
}

mtn_status mtn_attend_decode_append(mtn_pool *P, int32_t layer, const void *k, const void *v,
                                    const void *q, void *out, float *lse, int32_t n_split,
                                    void *stream) {
    return guarded(P, [&]() -> mtn_status {
        mtn_status st = check_call(P, layer, stream);
        if (st) return st;
        if (bad_buf(k) || bad_buf(v) || bad_buf(q) || bad_buf(out))
            return fail(P, MTN_ERR_INVALID_ARG, "null or misaligned k, v, q or out");
        if (!P->all_single) return fail(P, MTN_ERR_BAD_STATE, "decode needs n_tok == 1 everywhere");
        if (n_split < 0 || n_split > kMaxSplit) return fail(P, MTN_ERR_INVALID_ARG, "bad n_split");
        if (P->layer_done[layer]) return fail(P, MTN_ERR_BAD_STATE, "layer already appended");
        return decode_impl(P, layer, q, out, lse, n_split, stream, k, v);
    });
}

mtn_status mtn_attend_decode_noalloc(mtn_pool *P, int32_t layer, const void *q, void *out,
                                     float *lse, int32_t n_split, void *stream) {
    return guarded(P, [&]() -> mtn_status {
        mtn_status st = check_call(P, layer, stream);
        if (st) return st;
        if (bad_buf(q) || bad_buf(out)) return fail(P, MTN_ERR_INVALID_ARG, "null or misaligned q or out");
        if (!P->all_single) return fail(P, MTN_ERR_BAD_STATE, "decode needs n_tok == 1 everywhere");
        if (n_split < 0 || n_split > kMaxSplit) return fail(P, MTN_ERR_INVALID_ARG, "bad n_split");
        if (!P->layer_done[layer]) return fail(P, MTN_ERR_BAD_STATE, "layer not appended");
        const size_t per_split = (size_t)P->T * P->cfg.n_q_heads * (P->cfg.head_dim + 2);
        if (n_split == 0) {
            // the automatic split, reduced to what the static workspace holds
            n_split = auto_split(P, P->T);
            while (n_split > 1 && per_split * n_split > P->scratch_floats) --n_split;
        } else if (n_split > 1 && per_split * n_split > P->scratch_floats) {
            return fail(P, MTN_ERR_INVALID_ARG,
                        "split partials exceed the static workspace (4 Mi floats)");
        }
        return decode_impl(P, layer, q, out, lse, n_split, stream, nullptr, nullptr, P->d_scratch,
                           P->scratch_floats);
    });
}

mtn_status mtn_frame_step(mtn_pool *P, const mtn_frame_batch *b, void *stream) {
    return guarded(P, [&]() -> mtn_status {
        if (!P || !b) return MTN_ERR_INVALID_ARG;
        if (P->plan_open) return fail(P, MTN_ERR_BAD_STATE, "a plan is already open");
        const int32_t n = b->n_seq;
        if (n < 1 || n > P->cfg.max_sessions || !b->sids || !b->chunk_len || !b->n_decode)
            return fail(P, MTN_ERR_INVALID_ARG, "bad batch");
        if (!P->host_only && (bad_buf(b->q_chunk) || bad_buf(b->k_chunk) || bad_buf(b->v_chunk) ||
                              bad_buf(b->out_chunk)))
            return fail(P, MTN_ERR_INVALID_ARG, "null or misaligned chunk buffer");
        if (b->n_split < 0 || b->n_split > kMaxSplit) return fail(P, MTN_ERR_INVALID_ARG, "bad n_split");
        int32_t max_dec = 0;
        int64_t Tc = 0;
        std::vector<uint8_t> seen((size_t)P->cfg.max_sessions, 0);
        for (int32_t i = 0; i < n; ++i) {
            int32_t sid = b->sids[i];
            if (sid < 0 || sid >= P->cfg.max_sessions || !P->is_open[sid])
                return fail(P, MTN_ERR_BAD_SESSION, "session not open");
            if (seen[sid]) return fail(P, MTN_ERR_INVALID_ARG, "duplicate session in batch");
            seen[sid] = 1;
            if (b->chunk_len[i] < 1) return fail(P, MTN_ERR_INVALID_ARG, "chunk_len < 1");
            if (b->chunk_len[i] > P->cfg.max_chunk)
                return fail(P, MTN_ERR_CHUNK_TOO_LARGE, "chunk_len > max_chunk");
            if (b->n_decode[i] < 0) return fail(P, MTN_ERR_INVALID_ARG, "n_decode < 0");
            if (P->unbounded && P->len[sid] + b->chunk_len[i] + b->n_decode[i] > P->cfg.max_len)
                return fail(P, MTN_ERR_SESSION_FULL, "frame would pass max_len");
            max_dec = std::max(max_dec, b->n_decode[i]);
            Tc += b->chunk_len[i];
        }
        if (!P->host_only && max_dec > 0 &&
            (bad_buf(b->q_dec) || bad_buf(b->k_dec) || bad_buf(b->v_dec) || bad_buf(b->out_dec)))
            return fail(P, MTN_ERR_INVALID_ARG, "null or misaligned decode buffer");
        {   // whole-frame capacity check before any launch
            std::vector<uint8_t> lbseen((size_t)P->row_len, 0);
            int64_t need = 0;
            for (int32_t i = 0; i < n; ++i)
                need += new_blocks_needed(P, b->sids[i], P->len[b->sids[i]],
                                          (int64_t)b->chunk_len[i] + b->n_decode[i], lbseen);
            if (need > P->alloc.n_free()) return fail(P, MTN_ERR_POOL_EXHAUSTED, "pool exhausted");
        }
        // the decode rounds' batches, allocated before anything changes
        std::vector<int32_t> sids, ones, rows;
        sids.reserve((size_t)n);
        ones.reserve((size_t)n);
        rows.reserve((size_t)n);
        // From here on an error abandons the open plan (mtn_plan_abort); plans
        // of this frame that already committed stay committed.
        mtn_status st = frame_plans(P, b, stream, Tc, max_dec, sids, ones, rows);
        if (st && P->plan_open) plan_abort_impl(P);
        return st;
    });
}

mtn_status mtn_pool_stats(const mtn_pool *P, mtn_pool_stats_t *out) {
    if (!P || !out) return MTN_ERR_INVALID_ARG;
    out->capacity = P->cfg.n_blocks;
    out->assigned = P->assigned;
    out->reserved = P->unbounded ? P->assigned : P->reserved;
    out->open_sessions = P->n_open;
    out->blocks_per_session = P->row_len;
    out->ring_tokens = P->R;
    out->sink_blocks = P->nsb;
    return MTN_OK;
}

mtn_status mtn_session_info(const mtn_pool *P, int32_t sid, int64_t *len, int32_t *n_assigned) {
    if (!P) return MTN_ERR_INVALID_ARG;
    if (sid < 0 || sid >= P->cfg.max_sessions || !P->is_open[sid]) return MTN_ERR_BAD_SESSION;
    if (len) *len = P->len[sid];
    if (n_assigned) *n_assigned = P->n_assigned[sid];
    return MTN_OK;
}

mtn_status mtn_session_block_table(const mtn_pool *P, int32_t sid, int32_t *out, int32_t cap,
                                   int32_t *n_out) {
    if (!P || !out) return MTN_ERR_INVALID_ARG;
    if (sid < 0 || sid >= P->cfg.max_sessions || !P->is_open[sid]) return MTN_ERR_BAD_SESSION;
    if (cap < P->row_len) return MTN_ERR_INVALID_ARG;
    std::memcpy(out, &P->table[(size_t)sid * P->row_len], sizeof(int32_t) * P->row_len);
    if (n_out) *n_out = P->row_len;
    return MTN_OK;
}

mtn_status mtn_plan_info(const mtn_pool *P, int64_t *pos, int32_t *block, int32_t *offset,
                         int32_t cap, int64_t *ev_lo, int64_t *ev_hi, int32_t *n_tok_out) {
    if (!P) return MTN_ERR_INVALID_ARG;
    if (!P->plan_open) return MTN_ERR_BAD_STATE;
    if ((pos || block || offset) && cap < P->T) return MTN_ERR_INVALID_ARG;
    if ((ev_lo || ev_hi) && cap < P->n_seq) return MTN_ERR_INVALID_ARG;
    for (int32_t t = 0; t < P->T; ++t) {
        if (pos) pos[t] = P->tok_pos[t];
        if (block) block[t] = P->tok_block[t];
        if (offset) offset[t] = P->tok_off[t];
    }
    for (int32_t i = 0; i < P->n_seq; ++i) {
        int64_t lo = 0, hi = 0;
        if (!P->unbounded) {
            int64_t L0 = P->seq_pos0[i];
            lo = std::max<int64_t>(P->S, L0 - P->W);
            hi = std::max<int64_t>(lo, L0 + P->seq_ntok[i] - P->W);
        }
        if (ev_lo) ev_lo[i] = lo;
        if (ev_hi) ev_hi[i] = hi;
    }
    if (n_tok_out) *n_tok_out = P->T;
    return MTN_OK;
}

mtn_status mtn_debug_poison_dead(mtn_pool *P, void *stream) {
    return guarded(P, [&]() -> mtn_status {
        if (!P) return MTN_ERR_INVALID_ARG;
        if (P->host_only) return fail(P, MTN_ERR_BAD_STATE, "host-only pool has no device path");
        if (P->plan_open) return fail(P, MTN_ERR_BAD_STATE, "plan open");
        // live[b] bit o set <=> slot o of block b holds a retained position
        std::vector<uint16_t> live((size_t)P->cfg.n_blocks, 0);
        for (int32_t sid = 0; sid < P->cfg.max_sessions; ++sid) {
            if (!P->is_open[sid]) continue;
            const int32_t *row = &P->table[(size_t)sid * P->row_len];
            int64_t L = P->len[sid];
            int64_t lo = P->unbounded ? 0 : std::max<int64_t>(P->S, L - P->W);
            auto mark = [&](int64_t p) {
                int32_t lb, off;
                logical_slot(P, p, &lb, &off);
                if (row[lb] >= 0) live[(size_t)row[lb]] |= (uint16_t)(1u << off);
            };
            for (int64_t p = 0; p < std::min<int64_t>(P->S, L); ++p) mark(p);
            for (int64_t p = lo; p < L; ++p) mark(p);
        }
        hipStream_t s = (hipStream_t)stream;
        uint16_t *d_live = nullptr;
        HIP_TRY(P, hipMalloc(&d_live, sizeof(uint16_t) * live.size()));
        HIP_TRY(P, hipMemcpy(d_live, live.data(), sizeof(uint16_t) * live.size(),
                             hipMemcpyHostToDevice));
        if (P->cfg.kv_dtype == MTN_FP8_E4M3)
            HIP_TRY(P, launch_poison_fp8(geom(P), P->cfg.n_layers, P->cfg.n_blocks, d_live, s));
        else
            HIP_TRY(P, launch_poison(P->cfg.kv_dtype, geom(P), P->cfg.n_layers, P->cfg.n_blocks, d_live, s));
        HIP_TRY(P, hipStreamSynchronize(s));
        HIP_TRY(P, hipFree(d_live));
        return MTN_OK;
    });
}

mtn_status mtn_pool_set_prefill_pass_rows(mtn_pool *P, int32_t rows) {
    return guarded(P, [&]() -> mtn_status {
        if (!P) return MTN_ERR_INVALID_ARG;
        if (rows != 0 && !prefill_pass_rows_valid(rows))
            return fail(P, MTN_ERR_INVALID_ARG, "prefill pass rows must be 0, 128 or 256");
        P->pf_rows_cfg = rows;
        return MTN_OK;
    });
}

mtn_status mtn_pool_set_decode_kernel(mtn_pool *P, int32_t kind) {
    return guarded(P, [&]() -> mtn_status {
        if (!P) return MTN_ERR_INVALID_ARG;
        if (kind < 0 || kind > 2) return fail(P, MTN_ERR_INVALID_ARG, "kind must be 0, 1 or 2");
        if (P->plan_open) return fail(P, MTN_ERR_BAD_STATE, "plan open");
        const mtn_pool_config &c = P->cfg;
        if (kind == 1 && c.kv_dtype == MTN_FP8_E4M3)
            return fail(P, MTN_ERR_UNSUPPORTED, "the FP8 cache has no vector decode kernel");
        if (kind == 2 && c.kv_dtype == MTN_F32)
            return fail(P, MTN_ERR_UNSUPPORTED, "fp32 pools have no matrix decode kernel");
        if (kind == 2 && !attn_mfma_bf16_supported(c.head_dim, P->G))
            return fail(P, MTN_ERR_UNSUPPORTED, "no matrix decode kernel for this shape");
        P->decode_kernel = kind;
        if (!P->host_only) P->resident_units = count_resident_units(P);
        return MTN_OK;
    });
}

mtn_status mtn_pool_last_split(const mtn_pool *P, int32_t *n_split) {
    if (!P || !n_split) return MTN_ERR_INVALID_ARG;
    *n_split = P->last_split;
    return MTN_OK;
}

mtn_status mtn_debug_inject_failure(mtn_pool *P, int64_t launch_index) {
    if (!P || launch_index < -1) return MTN_ERR_INVALID_ARG;
    P->fail_at = launch_index;
    return MTN_OK;
}

mtn_status mtn_pool_set_timing(mtn_pool *P, int32_t enable) {
    return guarded(P, [&]() -> mtn_status {
        if (!P) return MTN_ERR_INVALID_ARG;
        P->timing = enable != 0;
        return MTN_OK;
    });
}

mtn_status mtn_pool_kernel_times(mtn_pool *P, int64_t *launches, double *ms) {
    return guarded(P, [&]() -> mtn_status {
        if (!P || !launches || !ms) return MTN_ERR_INVALID_ARG;
        for (int c = 0; c < 4; ++c) {
            for (auto &pr : P->ev_open[c]) {
                HIP_TRY(P, hipEventSynchronize(pr.b));
                float t = 0.f;
                HIP_TRY(P, hipEventElapsedTime(&t, pr.a, pr.b));
                P->t_ms[c] += t;
                P->t_launch[c]++;
                P->ev_spare.push_back(pr.a);
                P->ev_spare.push_back(pr.b);
            }
            P->ev_open[c].clear();
            launches[c] = P->t_launch[c];
            ms[c] = P->t_ms[c];
            P->t_launch[c] = 0;
            P->t_ms[c] = 0.0;
        }
        return MTN_OK;
    });
}

mtn_status mtn_hbm_read(const void *src, size_t bytes, void *stream) {
    if (!src || (bytes % 8192) || ((uintptr_t)src % 16)) return MTN_ERR_INVALID_ARG;
    hipError_t e = launch_read(src, bytes, nullptr, (hipStream_t)stream);
    return e == hipSuccess ? MTN_OK : MTN_ERR_DEVICE;
}

mtn_status mtn_hbm_copy(const void *src, void *dst, size_t bytes, void *stream) {
    if (!src || !dst || (bytes % 16) || ((uintptr_t)src % 16) || ((uintptr_t)dst % 16))
        return MTN_ERR_INVALID_ARG;
    hipError_t e = launch_copy(src, dst, bytes, (hipStream_t)stream);
    return e == hipSuccess ? MTN_OK : MTN_ERR_DEVICE;
}

}  // extern "C"
