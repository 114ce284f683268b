// C ABI of libnld: host-side validation, workspace layout and launch sequence of
// the block-decode step (declared in include/nld.h).
#include "../../include/nld.h"
#include "nld_internal.h"

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

using namespace nld;

struct nld_model {
    nld_config cfg;
    nld_weights w;
    std::vector<nld_layer_weights> layers;
};

namespace {

thread_local char g_err[512] = "";

nld_status fail(nld_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return st;
}

#define HIP_TRY(expr)                                                                              \
    do {                                                                                           \
        hipError_t e_ = (expr);                                                                    \
        if (e_ != hipSuccess) return fail(NLD_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_)); \
    } while (0)

// ---------------------------------------------------------------- tracing aid
// While tracing is on, every launch inside a TraceScope gets its own pair of events,
// recorded by the launch on its own dispatch (kernel start and end), filed under the
// scope's kernel class.
struct TraceRec {
    int cls;
    bool first;   // first launch of its scope: the scope counts once in its class
    hipEvent_t start, stop;
};
bool g_trace_on = false;
std::vector<TraceRec> g_trace;
thread_local int g_trace_cls = -1;
thread_local bool g_trace_scope_new = false;

struct TraceScope {
    int saved;
    TraceScope(int cls, hipStream_t) : saved(g_trace_cls) {
        g_trace_cls = cls;
        g_trace_scope_new = true;
    }
    ~TraceScope() { g_trace_cls = saved; }
};

int device_cus();

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
inline int cdiv(int a, int b) { return (a + b - 1) / b; }

int env_int(const char* name, int dflt) {
    const char* v = getenv(name);
    return (v && *v) ? atoi(v) : dflt;
}

// Operand sites carried in plain bf16 instead of split form: NLD_PLAIN_SITES, a comma-separated list
// of norm, final, q, kv, p, o, act (precision knob; default: none, every site split).
uint32_t plain_sites() {
    const char* v = getenv("NLD_PLAIN_SITES");
    if (!v || !*v) return 0u;
    static const struct { const char* name; uint32_t bit; } names[] = {
        {"norm", SITE_NORM}, {"final", SITE_FINAL}, {"q", SITE_Q}, {"kv", SITE_KV},
        {"p", SITE_P}, {"o", SITE_O}, {"act", SITE_ACT}};
    uint32_t m = 0u;
    for (const auto& n : names) {
        const size_t len = strlen(n.name);
        for (const char* c = v; (c = strstr(c, n.name)) != nullptr; c += len) {
            const bool start = c == v || c[-1] == ',';
            const bool end = c[len] == '\0' || c[len] == ',';
            if (start && end) m |= n.bit;
        }
    }
    return m;
}

}  // namespace

bool nld::trace_launch_events(hipEvent_t* start, hipEvent_t* stop) {
    if (!g_trace_on || g_trace_cls < 0) return false;
    TraceRec r{};
    r.cls = g_trace_cls;
    r.first = g_trace_scope_new;
    g_trace_scope_new = false;
    if (hipEventCreate(&r.start) != hipSuccess) return false;
    if (hipEventCreate(&r.stop) != hipSuccess) {
        (void)hipEventDestroy(r.start);
        return false;
    }
    g_trace.push_back(r);
    *start = r.start;
    *stop = r.stop;
    return true;
}

namespace {

// ---------------------------------------------------------------- workspace layout
struct Layout {
    int M, Mpad, units, n_splits, chunk, row_tiles, attn_kh, attn_z, n_parts, rows_pad, lm_tiles, lm_parts;
    bool attn_items;         // length-aware attention work (batches)
    int n_sk_ctr, sk_ctr0;   // split-K residual GEMM: counters (one per column group) from tile counter sk_ctr0
    int n_nk_ctr, nk_ctr0;   // normed GEMM of 17..64 rows: counters (one per column tile) from tile counter nk_ctr0
    int n_tk_ctr, tk_ctr0;   // tiled GEMM with K slices (M > 64): counters (one per tile group) from tk_ctr0
    int tk_part_wgs;         // (tile group, slice) partials its buffer holds
    size_t nk_part_floats;   // and the size of its partials buffer
    size_t status, x, xg, part_ss, q, o, act, keys, lse, rope, po, pml, blk_k, blk_v, tile_ctr, sk_part, tk_part, lora_t, drafts,
        ens_logits, ens_v, nk_part, total;
};

// k: block rows per sequence.  quad_k > 0: the block is a quadratic self-speculation layout
// with chain length quad_k (k = quad_k * (quad_k + 1)), which adds the ensemble verifier's buffers.
Layout make_layout(const nld_config& c, int batch, int k, int max_len, int quad_k = 0) {
    Layout L{};
    L.M = batch * k;
    // operand rows: whole 64-row groups, or whole 128-row tiles of the tiled GEMM (M > 64)
    L.Mpad = L.M > 64 ? cdiv(L.M, gemm_tile_row_pad()) * gemm_tile_row_pad() : cdiv(L.M, 64) * 64;
    L.units = batch * c.n_kv_heads;
    const int G = c.n_q_heads / c.n_kv_heads;
    L.row_tiles = cdiv(G * k, 16);
    L.attn_kh = L.row_tiles <= 4 ? 2 : 1;          // wavefronts per row tile (each takes half of a stage's keys)
    L.attn_z = cdiv(L.row_tiles, 8 / L.attn_kh);
    L.rows_pad = L.attn_z * (8 / L.attn_kh) * 16;
    L.lm_tiles = cdiv(c.vocab, 16);
    L.lm_parts = L.lm_tiles;  // upper bound on argmax partials per row (one per LM-head workgroup)
    // key splits: aim for about `target` workgroups, chunks a multiple of 64 keys.  One
    // workgroup per CU while there are few (unit, row slice) pairs (batch 1: each workgroup
    // is then a short latency chain); up to four per CU when there are many, so that long
    // and ragged key ranges are cut finer than one per CU.
    // With more than one sequence the workgroups take length-aware items (only splits holding
    // committed keys get a workgroup), so the splits may be cut finer: with one row slice the plan
    // aims at NLD_ATTN_ITEMS_FINER (default 2) times as many workgroups as it would at max_len.
    // (Measured: 8B batch 32, ragged prefixes, one slice: 198 us against 214 us at 1x and 254 us
    // without items; 14B batch 8, equal prefixes, two slices: 2x 366 us against 341 us at 1x.)
    L.attn_items = batch > 1 && !env_int("NLD_ATTN_NO_ITEMS", 0);
    const int pairs = L.units * L.attn_z;
    const int finer = L.attn_items ? env_int("NLD_ATTN_ITEMS_FINER", L.attn_z == 1 ? 2 : 1) : 1;
    const int target = env_int("NLD_ATTN_TARGET_WG", finer * device_cus() * std::min(4, std::max(1, pairs / 16)));
    int ns = target / (L.units * L.attn_z) - 1;    // one workgroup per (unit, row slice) is the block part
    const int max_splits = cdiv(max_len, 64);
    if (ns > max_splits) ns = max_splits;
    if (ns > 255) ns = 255;   // the merge handles up to 256 partials per row
    if (ns < 1) ns = 1;
    L.chunk = cdiv(cdiv(max_len, ns), 64) * 64;
    L.n_splits = cdiv(max_len, L.chunk);
    L.n_parts = L.n_splits + 1;   // prefix splits + the block part (key halves merge inside the workgroup)

    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off = align256(off + bytes);
        return o;
    };
    const size_t H = c.hidden, QD = (size_t)c.n_q_heads * c.head_dim;
    L.status = take(4);
    L.x = take(4 * L.Mpad * H);
    L.xg = take(4 * L.Mpad * H);   // split operand (hi and lo bf16)
    L.part_ss = take(4 * L.Mpad * (H / 16));
    // q, o and act are split operands too: 4 bytes per value
    L.q = take(4 * std::max(L.Mpad * QD, (size_t)L.units * L.row_tiles * 16 * c.head_dim));
    L.o = take(4 * L.Mpad * QD);
    L.act = take(4 * L.Mpad * (size_t)cdiv(c.ffn, 32) * 32);
    L.keys = take(8 * L.Mpad * (size_t)L.lm_parts);
    L.lse = take(8 * L.Mpad * (size_t)L.lm_parts);   // softmax statistics per argmax partial (denoising)
    L.rope = take(8 * L.Mpad * (size_t)(c.head_dim / 2));
    // split-K GEMM (M <= 64; the O, down, QKV and gate/up projections): one counter per column
    // group of at least 2 tiles of the O, down and QKV projections, and the partials of up to
    // SPLITK_MAX slices (gate/up, with more tiles, runs unsplit)
    const int sk_tiles = std::max((int)H / 16, (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim / 16);
    L.n_sk_ctr = L.M <= 64 ? cdiv(sk_tiles, 2) : 0;
    const int sk_rows = L.M <= 32 ? 32 : 64;
    L.sk_ctr0 = 2 * c.n_layers + 1;
    // normed GEMM of 17..64 rows: one counter per column tile of the widest normed projection,
    // partials of every K slice
    const int nk_tiles = std::max(std::max(cdiv(c.vocab, 16), cdiv(c.ffn, 8)),
                                  (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim / 16);
    const bool nk = L.M > 16 && L.M <= 64;
    L.n_nk_ctr = nk ? nk_tiles : 0;
    L.nk_ctr0 = L.sk_ctr0 + L.n_sk_ctr;
    // per pass: QKV and gate/up of every layer, LM head; then the split-K counters and the
    // 17..64-row counters (all zeroed by the embedding kernel at the start of a pass)
    // tiled GEMM (M > 64) with K slices: one counter per 128 x 128 tile group of the widest
    // projection it may split (O, down, QKV, gate/up), partials of up to two workgroups per CU
    const bool tk = L.M > 64;
    L.n_tk_ctr = tk ? std::max(gemm_tile_groups(L.M, std::max(sk_tiles, cdiv(c.ffn, 8))), 1) : 0;
    L.tk_ctr0 = L.nk_ctr0 + L.n_nk_ctr;
    L.tk_part_wgs = tk ? 2 * gemm_tile_wgs_per_cu() * device_cus() : 0;
    // per pass: QKV and gate/up of every layer, LM head; then the split-K counters, the 17..64-row
    // counters and the tiled GEMM's counters (all zeroed by the embedding kernel at the start of a
    // pass; the split GEMMs also reset theirs after each use)
    L.tile_ctr = take(4 * (size_t)(2 * c.n_layers + 1 + L.n_sk_ctr + L.n_nk_ctr + L.n_tk_ctr));
    L.tk_part = take(4 * (size_t)L.tk_part_wgs * gemm_tile_part_floats_per_wg());
    // (the normed projections, LM head, QKV and gate/up, all reduce over hidden)
    L.nk_part_floats = nk ? (size_t)nk_tiles * cdiv(cdiv((int)H, 32), gemm_normk_kstep_span(L.M)) *
                                (L.M > 32 ? 4 : 2) * 256
                          : 0;
    L.nk_part = take(4 * L.nk_part_floats);
    // partials: whole column groups (at most 2 * n_sk_ctr + 4 tiles of 16) x sk_rows rows x slices
    L.sk_part = take(L.M <= 64 ? 4 * (size_t)(2 * L.n_sk_ctr + 4) * 16 * sk_rows * SPLITK_MAX : 0);
    L.po = take(4 * (size_t)L.units * L.n_parts * L.rows_pad * c.head_dim);
    L.pml = take(4 * 2 * (size_t)L.units * L.n_parts * L.rows_pad);
    L.blk_k = take(2 * (size_t)L.units * 2 * 64 * c.head_dim);   // block K/V, split: [unit][hi, lo][64][D]
    L.blk_v = take(2 * (size_t)L.units * 2 * 64 * c.head_dim);
    L.lora_t = take(4 * (size_t)L.Mpad * c.lora_rank);   // split lora_scale * (A o), draft passes only
    L.drafts = take(4 * (size_t)batch * k);              // nld_decode_steps: one step's drafts
    // quadratic self-speculation: the verifier rows' logits [batch][2 quad_k][vocab] and the ensemble's
    // argmax keys [batch][quad_k][ENS_CHUNKS]
    L.ens_logits = take(4 * (size_t)batch * 2 * quad_k * c.vocab);
    L.ens_v = take(8 * (size_t)batch * quad_k * ENS_CHUNKS);
    L.total = off;
    return L;
}

template <typename T>
T* at(void* ws, size_t off) { return (T*)((char*)ws + off); }

nld_status check_config(const nld_config* c) {
    if (!c) return fail(NLD_ERR_INVALID_ARG, "config is NULL");
    if (c->n_layers < 1 || c->hidden < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1 || c->ffn < 1 || c->vocab < 1)
        return fail(NLD_ERR_INVALID_ARG, "config sizes must be positive");
    if (c->hidden % 32) return fail(NLD_ERR_SHAPE, "hidden (%d) must be a multiple of 32", c->hidden);
    if (c->head_dim != 64 && c->head_dim != 128) return fail(NLD_ERR_SHAPE, "head_dim must be 64 or 128");
    if (c->n_q_heads % c->n_kv_heads) return fail(NLD_ERR_SHAPE, "n_q_heads must be a multiple of n_kv_heads");
    if (c->ffn % 8) return fail(NLD_ERR_SHAPE, "ffn (%d) must be a multiple of 8", c->ffn);
    if (c->mask_token_id < 0 || c->mask_token_id >= c->vocab)
        return fail(NLD_ERR_INVALID_ARG, "mask_token_id outside [0, vocab)");
    if (!(c->rope_base > 1.0f) || !(c->rms_eps >= 0.0f)) return fail(NLD_ERR_INVALID_ARG, "bad rope_base or rms_eps");
    if (c->lora_rank < 0 || !(fabsf(c->lora_scale) < INFINITY))
        return fail(NLD_ERR_INVALID_ARG, "lora_rank must be >= 0 and lora_scale finite");
    if (c->lora_rank % 32) return fail(NLD_ERR_SHAPE, "lora_rank (%d) must be a multiple of 32", c->lora_rank);
    if (c->lora_rank > 512) return fail(NLD_ERR_SHAPE, "lora_rank (%d) must be at most 512", c->lora_rank);
    return NLD_OK;
}

// ---------------------------------------------------------------- GEMM launch plans
// Normed multi-tile GEMM: k-steps per wavefront and wavefront count with ks * waves == ksteps.
bool plan_norm(int epi, int M, int ksteps, int* ks, int* waves) {
    if (M > 16 || env_int("NLD_NO_NORM_GEMM", 0)) return false;
    // k-steps per wavefront: 16 (8 wavefronts) where the epilogue needs registers, 8 (16 wavefronts) for SwiGLU
    const int pref = env_int(epi == EPI_QKV ? "NLD_NORM_KS_QKV" : epi == EPI_SWIGLU ? "NLD_NORM_KS_GU" : "NLD_NORM_KS_LM",
                             epi == EPI_SWIGLU ? 8 : 16);
    const int cand[] = {pref, 8, 16, 20, 4};
    for (int c : cand) {
        if (gemm_norm_supported(c) && ksteps % c == 0 && ksteps / c >= 1 && ksteps / c <= gemm_norm_max_waves(c)) {
            *ks = c;
            *waves = ksteps / c;
            return true;
        }
    }
    return false;
}

// Compute units of the current device (queried once per device; NLD_CUS overrides).
int device_cus() {
    const int forced = env_int("NLD_CUS", 0);
    if (forced > 0) return forced;
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cached[dev] == 0) {
        int n = 0;
        cached[dev] = (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
                          ? n : 256;
    }
    return cached[dev];
}

// Workgroups of the normed GEMM: one per CU, but at least two tiles per workgroup on
// average (each workgroup loads the whole operand once); tiles beyond the first one per
// workgroup are handed out dynamically.
// NLD_NORM_TPW_QKV / _GU / _LM: tiles per workgroup to aim for instead of 2.
int norm_grid(int epi, int n_tiles) {
    const int cus = device_cus();
    const int tpw = std::max(1, env_int(epi == EPI_QKV ? "NLD_NORM_TPW_QKV" : epi == EPI_SWIGLU ? "NLD_NORM_TPW_GU"
                                                                                                : "NLD_NORM_TPW_LM", 2));
    const int want = (n_tiles + tpw - 1) / tpw;
    return want < cus ? want : cus;
}

struct StreamPlan {
    int mt, ct, nw, gx, gy;
};

StreamPlan plan_stream(int epi, int M, int n_tiles) {
    StreamPlan p;
    p.mt = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
    p.gy = cdiv(M, 16 * p.mt);
    if (epi == EPI_LMHEAD) {
        p.ct = 4;
        p.nw = 4;
    } else if (epi == EPI_SWIGLU) {
        p.ct = 2;
        p.nw = 8;
    } else {
        // O and down on this kernel at up to 16 rows: 16 wavefronts with every load of their 8 k-steps in
        // flight (O at the 8B shapes: 10.8-11.0 against 11.2 us with 8 wavefronts)
        p.ct = 1;
        p.nw = epi == EPI_RESID && M <= 16 ? env_int("NLD_STREAM_NW_RESID", 16) : 8;
    }
    p.gx = cdiv(n_tiles, p.ct);
    return p;
}

enum Source { SRC_TOKENS = 0, SRC_DRAFT = 1, SRC_VERIFY = 2, SRC_QUAD = 3 };

struct PassIO {
    int source;
    const int32_t* tokens;
    const int32_t* anchor;
    const int32_t* draft_in;
    int mode, bidir_from;
    float* logits;
    int32_t* argmax_out;
    int finish;
    int32_t* draft_out;
    int32_t* accept_len;
    int32_t* committed;
    int32_t* next_anchor;
    bool advance_lengths;
    // denoising step / refresh
    int32_t* block;
    float threshold;
    int32_t* n_committed;
    int32_t* n_masked;
    float* conf_out;
    bool kv_only;   // refresh: stop after the last layer's K/V (no attention, FFN or LM head after it)
    // quadratic self-speculation (mode NLD_MODE_QUAD_INTERNAL): chain length and the verifier's mixture
    int quad_k;
    float lambda;
};

// Attention mode of a quadratic pass (never a caller's mode value).
constexpr int NLD_MODE_QUAD_INTERNAL = 2;

nld_status validate_call(const nld_model* m, const nld_kv_cache* kv, int batch, int k, void* ws, size_t ws_bytes,
                         Layout* out, int quad_k = 0) {
    if (!m) return fail(NLD_ERR_INVALID_ARG, "model is NULL");
    if (!kv || !kv->k || !kv->v || !kv->lengths) return fail(NLD_ERR_INVALID_ARG, "kv cache or one of its pointers is NULL");
    if (!ws) return fail(NLD_ERR_INVALID_ARG, "workspace is NULL");
    if (batch < 1) return fail(NLD_ERR_INVALID_ARG, "batch must be >= 1");
    if (kv->batch != batch) return fail(NLD_ERR_INVALID_ARG, "kv->batch (%d) != batch (%d)", kv->batch, batch);
    if (k < 1 || k > 64) return fail(NLD_ERR_INVALID_ARG, "k must be in [1, 64] (got %d)", k);
    if (kv->max_len < 64 || kv->max_len % 64) return fail(NLD_ERR_INVALID_ARG, "max_len must be a positive multiple of 64");
    const nld_config& c = m->cfg;
    const int G = c.n_q_heads / c.n_kv_heads;
    if (G * k > 256) return fail(NLD_ERR_SHAPE, "(n_q_heads/n_kv_heads)*k = %d exceeds 256", G * k);
    *out = make_layout(c, batch, k, kv->max_len, quad_k);
    if (ws_bytes < out->total)
        return fail(NLD_ERR_CAPACITY, "workspace holds %zu bytes, this call needs %zu", ws_bytes, out->total);
    return NLD_OK;
}

// The tiled GEMM takes every projection with more than 64 rows whose shape it supports.
bool use_tile(const GemmArgs& g) {
    return !env_int("NLD_NO_TILE_GEMM", 0) && !g.W2 && gemm_tile_supported(g.M, g.K, g.ksteps);
}

enum SplitKind { SK_O = 0, SK_DOWN = 1, SK_QKV = 2, SK_GU = 3 };

// K slices of the tiled GEMM (M > 64): enough slices to fill every CU's workgroup slots when the
// 128 x 128 tile groups alone leave CUs idle (O, down and QKV at a few hundred rows; gate/up has
// several groups per CU already), each slice at least two stages of 64 k.
// NLD_TILE_KSPLIT_<O|DOWN|QKV|GU> overrides the count (1: off).
int plan_tile_ksplit(int kind, const GemmArgs& g, const Layout& L) {
    static const char* names[] = {"NLD_TILE_KSPLIT_O", "NLD_TILE_KSPLIT_DOWN", "NLD_TILE_KSPLIT_QKV",
                                  "NLD_TILE_KSPLIT_GU"};
    const int groups = gemm_tile_groups(g.M, g.n_tiles);
    int ks = kind == SK_GU ? 1 : std::max(1, gemm_tile_wgs_per_cu() * device_cus() / groups);
    ks = env_int(names[kind], ks);
    ks = std::min(ks, std::min(gemm_tile_stages(g.ksteps) / 2, 8));
    if (ks <= 1 || groups > L.n_tk_ctr || groups * ks > L.tk_part_wgs) return 1;
    return ks;
}

hipError_t tile_gemm(int kind, int epi, const GemmArgs& g, void* ws, const Layout& L, hipStream_t s) {
    const int ks = epi == EPI_LMHEAD ? 1 : plan_tile_ksplit(kind, g, L);
    if (ks == 1) return launch_gemm_tile(epi, g, 1, nullptr, nullptr, s);
    return launch_gemm_tile(epi, g, ks, at<float>(ws, L.tk_part), at<unsigned>(ws, L.tile_ctr) + L.tk_ctr0, s);
}

// Split-K plan of a projection with at most 64 rows: ct column tiles per workgroup and
// ksplit K slices, so that column groups x slices is at most one workgroup per CU, with
// every wavefront (8 per workgroup) getting at least two k-steps.  Defaults per
// projection (measured on MI355X at the 8B shapes): up to 16 rows down 2 tiles, O off (the
// streamed GEMM, 11.3 against 12.9 us), QKV and gate/up off (the normed multi-tile kernel is
// faster there); 17..64 rows every projection 4 tiles, except QKV at 17..32 rows, 3 tiles (taken
// there before the normed multi-tile kernel).  Environment overrides:
// NLD_SPLITK_<O|DOWN|QKV|GU> = "ct,ksplit" ("ct,0": ksplit from the rule; "0": off),
// NLD_SPLITK / NLD_SPLITK_CT for every projection at once, NLD_NO_SPLITK = 1: off.

bool plan_splitk(int kind, int epi, const GemmArgs& g, const Layout& L, int* ct, int* ksplit) {
    if (g.W2 || L.n_sk_ctr == 0 || env_int("NLD_NO_SPLITK", 0)) return false;
    static const char* names[] = {"NLD_SPLITK_O", "NLD_SPLITK_DOWN", "NLD_SPLITK_QKV", "NLD_SPLITK_GU"};
    // column tiles per workgroup: up to 16 rows; 17..32 rows; 33..64 rows
    static const int dflt_ct[3][4] = {{0, 2, 0, 0}, {4, 4, 3, 4}, {4, 4, 4, 4}};
    int c = dflt_ct[g.M <= 16 ? 0 : (g.M <= 32 ? 1 : 2)][kind], ks = 0;
    const char* v = getenv(names[kind]);
    if (v && *v) {
        c = atoi(v);
        const char* comma = strchr(v, ',');
        ks = comma ? atoi(comma + 1) : 0;
    }
    c = env_int("NLD_SPLITK_CT", c);
    ks = env_int("NLD_SPLITK", ks);
    if (c <= 0 || !gemm_splitk_supported(epi, g.M, c)) return false;
    const int groups = cdiv(g.n_tiles, c);
    if (ks <= 0) ks = std::min(std::max(1, device_cus() / groups), std::max(1, g.ksteps / 16));
    if (groups > L.n_sk_ctr) ks = 1;   // no counters (and no partials) for that many groups
    *ct = c;
    *ksplit = std::max(1, std::min(std::min(ks, SPLITK_MAX), g.ksteps));
    return true;
}

// The multi-tile GEMM of 17..64 rows when it applies (counters and partials fit the
// workspace); returns false otherwise.
bool try_normk(int epi, GemmArgs& g, void* ws, const Layout& L, hipStream_t s, int* parts_out, hipError_t* err) {
    if (L.n_nk_ctr == 0 || !gemm_normk_supported(epi, g.M) || g.W2 || env_int("NLD_NO_NORMK", 0)) return false;
    const int slices = cdiv(g.ksteps, gemm_normk_kstep_span(g.M));
    if (g.n_tiles > L.n_nk_ctr || cdiv(g.n_tiles, gemm_normk_max_tiles()) * slices > L.lm_parts ||
        (size_t)g.n_tiles * slices * (g.M > 32 ? 4 : 2) * 256 > L.nk_part_floats)
        return false;
    // about one workgroup per CU; the LM head writes one argmax key per row and workgroup (at most
    // lm_parts per row)
    int gx = std::max(cdiv(g.n_tiles, gemm_normk_max_tiles()), std::max(1, device_cus() / slices));
    if (epi == EPI_LMHEAD) gx = std::min(gx, std::max(1, L.lm_parts / slices));
    g.n_parts = gx * slices;
    if (parts_out) *parts_out = g.n_parts;
    *err = launch_gemm_normk(epi, gx, g, at<float>(ws, L.nk_part), at<unsigned>(ws, L.tile_ctr) + L.nk_ctr0, s);
    return true;
}

// Residual projections (O, down): the tiled GEMM when it applies, the split-K GEMM for up to
// 64 rows, else the streamed one.  (The multi-tile GEMM of 17..64 rows with the residual
// epilogue was slower at 56 rows: down 60.5 against 35.1 us, its 12 K slices' partials
// dominating.)
hipError_t resid_gemm(int kind, const GemmArgs& g, void* ws, const Layout& L, hipStream_t s) {
    if (use_tile(g)) return tile_gemm(kind, EPI_RESID, g, ws, L, s);
    int ct = 0, ksplit = 0;
    if (plan_splitk(kind, EPI_RESID, g, L, &ct, &ksplit))
        return launch_gemm_splitk(EPI_RESID, ct, ksplit, g, at<float>(ws, L.sk_part),
                                  at<unsigned>(ws, L.tile_ctr) + L.sk_ctr0, s);
    StreamPlan p = plan_stream(EPI_RESID, g.M, g.n_tiles);
    if (g.W2) p.nw = 8;   // the second source's k-steps need the 8-wavefront kernel's registers
    return launch_gemm_stream(EPI_RESID, p.mt, p.ct, p.nw, p.gx, p.gy, g, s);
}

// One projection whose operand is RMSNorm(x) (QKV, gate/up, LM head): the normed
// multi-tile kernel for M <= 16, else the streamed kernel (both read the bf16
// operand and the row statistics the producer of x wrote).
hipError_t normed_gemm(int epi, GemmArgs g, void* ws, const Layout& L, hipStream_t s, int* parts_out) {
    g.A = at<uint16_t>(ws, L.xg);
    g.part_ss = at<float>(ws, L.part_ss);
    g.n_ss = g.K / 16;
    int ks = 0, waves = 0, ct = 0, ksplit = 0;
    hipError_t err = hipSuccess;
    // QKV of 17..32 rows: the split-K GEMM, 3 column tiles x 2 K slices per workgroup (8B shapes at
    // k = 32: 23.6 against 25.2 us for the multi-tile kernel)
    if (epi == EPI_QKV && g.M > 16 && g.M <= 32 && plan_splitk(SK_QKV, epi, g, L, &ct, &ksplit))
        return launch_gemm_splitk(epi, ct, ksplit, g, at<float>(ws, L.sk_part),
                                  at<unsigned>(ws, L.tile_ctr) + L.sk_ctr0, s);
    if (try_normk(epi, g, ws, L, s, parts_out, &err)) return err;   // 17..64 rows
    if ((epi == EPI_QKV || (epi == EPI_SWIGLU && g.M > 16)) &&
        plan_splitk(epi == EPI_QKV ? SK_QKV : SK_GU, epi, g, L, &ct, &ksplit))
        return launch_gemm_splitk(epi, ct, ksplit, g, at<float>(ws, L.sk_part),
                                  at<unsigned>(ws, L.tile_ctr) + L.sk_ctr0, s);
    if (plan_norm(epi, g.M, g.ksteps, &ks, &waves)) {
        const int grid = norm_grid(epi, g.n_tiles);
        if (parts_out) *parts_out = grid;
        g.n_parts = grid;
        return launch_gemm_norm(epi, ks, waves, grid, g, s);
    }
    if (use_tile(g)) {
        g.n_parts = gemm_tile_parts(g.n_tiles);
        if (parts_out) *parts_out = g.n_parts;
        return tile_gemm(epi == EPI_QKV ? SK_QKV : SK_GU, epi, g, ws, L, s);
    }
    const StreamPlan p = plan_stream(epi, g.M, g.n_tiles);
    if (parts_out) *parts_out = p.gx;
    g.n_parts = p.gx;
    return launch_gemm_stream(epi, p.mt, p.ct, p.nw, p.gx, p.gy, g, s);
}

nld_status run_pass(const nld_model* mdl, const nld_kv_cache* kv, int batch, int k, const PassIO& io, void* ws,
                    const Layout& L, hipStream_t s) {
    const nld_config& c = mdl->cfg;
    const int M = L.M;
    const int D = c.head_dim, nq = c.n_q_heads, nkv = c.n_kv_heads;
    const size_t kv_layer = (size_t)batch * nkv * kv->max_len * D;
    uint32_t* status = at<uint32_t>(ws, L.status);
    float* x = at<float>(ws, L.x);

    EmbedArgs e{};
    e.tokens = io.tokens;
    e.anchor = io.anchor;
    e.draft = io.draft_in;
    e.source = io.source;
    e.k_blk = k;
    e.M = M;
    e.mask_id = c.mask_token_id;
    e.vocab = c.vocab;
    e.hidden = c.hidden;
    e.embed = (const uint16_t*)mdl->w.embed;
    e.gain = (const uint16_t*)mdl->layers[0].attn_norm;
    e.x = x;
    e.xg = at<uint16_t>(ws, L.xg);
    e.part_ss = at<float>(ws, L.part_ss);
    e.status = status;
    e.rope = at<float2>(ws, L.rope);
    e.tile_ctr = at<unsigned>(ws, L.tile_ctr);
    e.n_tile_ctr = 2 * c.n_layers + 1 + L.n_sk_ctr + L.n_nk_ctr + L.n_tk_ctr;
    e.lengths = kv->lengths;
    e.max_len = kv->max_len;
    e.head_dim = c.head_dim;
    e.quad_k = io.quad_k;
    const uint32_t plain = plain_sites();
    e.plain = plain & SITE_NORM;
    for (int i = 0; i < c.head_dim / 2; ++i) e.inv_freq[i] = pow((double)c.rope_base, -2.0 * i / (double)c.head_dim);
    {
        TraceScope ts(NLD_TRACE_EMBED, s);
        HIP_TRY(launch_embed(e, s));
    }

    const int ks_h = cdiv(c.hidden, 32), ks_q = cdiv(nq * D, 32), ks_f = cdiv(c.ffn, 32);
    for (int l = 0; l < c.n_layers; ++l) {
        const nld_layer_weights& W = mdl->layers[l];
        uint16_t* kc = (uint16_t*)kv->k + (size_t)l * kv_layer;
        uint16_t* vc = (uint16_t*)kv->v + (size_t)l * kv_layer;

        GemmArgs g{};
        g.eps = c.rms_eps;
        g.M = M;
        g.K = c.hidden;
        g.W = (const uint4*)W.w_qkv;
        g.n_tiles = (nq + 2 * nkv) * D / 16;
        g.ksteps = ks_h;
        g.q_out = at<uint16_t>(ws, L.q);
        g.q_row_tiles = L.row_tiles;
        g.kc = kc;
        g.vc = vc;
        g.write_cache = io.mode == NLD_MODE_VERIFY || io.mode == NLD_MODE_QUAD_INTERNAL;   // quad: chain rows
        g.quad_k = io.quad_k;
        g.blk_k = at<uint16_t>(ws, L.blk_k);
        g.blk_v = at<uint16_t>(ws, L.blk_v);
        g.lengths = kv->lengths;
        g.k_blk = k;
        g.n_q_heads = nq;
        g.n_kv_heads = nkv;
        g.head_dim = D;
        g.max_len = kv->max_len;
        g.rope = at<float2>(ws, L.rope);
        g.tile_ctr = at<unsigned>(ws, L.tile_ctr) + 2 * l;
        g.status = status;
        g.plain = plain & (SITE_Q | SITE_KV);
        {
            TraceScope ts(NLD_TRACE_QKV, s);
            HIP_TRY(normed_gemm(EPI_QKV, g, ws, L, s, nullptr));
        }
        if (io.kv_only && l == c.n_layers - 1) break;   // every layer's K/V rows are written

        AttnArgs at_{};
        at_.q = at<uint16_t>(ws, L.q);
        at_.kc = kc;
        at_.vc = vc;
        at_.lengths = kv->lengths;
        at_.o = at<uint16_t>(ws, L.o);
        at_.blk_k = at<uint16_t>(ws, L.blk_k);
        at_.blk_v = at<uint16_t>(ws, L.blk_v);
        at_.part_o = at<float>(ws, L.po);
        at_.part_ml = at<float>(ws, L.pml);
        at_.k_blk = k;
        at_.n_q_heads = nq;
        at_.n_kv_heads = nkv;
        at_.max_len = kv->max_len;
        at_.n_splits = L.n_splits;
        at_.chunk = L.chunk;
        at_.mode = io.mode;
        at_.bidir_from = io.bidir_from;
        at_.rows_pad = L.rows_pad;
        at_.row_tiles = L.row_tiles;
        at_.quad_k = io.quad_k;
        at_.n_parts = L.n_parts;
        at_.items = L.attn_items ? 1 : 0;
        at_.n_seq = batch;
        at_.scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
        at_.plain = plain & (SITE_P | SITE_O);
        // Prefix stages 1 and 2 are requested once stage 0 is in LDS: requested with it, the three
        // stages of every workgroup arrive interleaved and stage 0 comes late (8B shapes, k = 16:
        // 16.55 against 17.43 us per attention and merge).  NLD_ATTN_LATE = 0 / 1: all at once /
        // stage 2 only.
        at_.late = env_int("NLD_ATTN_LATE", 2);
        {
            TraceScope ts(NLD_TRACE_ATTENTION, s);
            HIP_TRY(launch_attention(D, L.attn_kh, L.attn_z, L.units, at_, s));
            HIP_TRY(launch_attention_combine(D, L.units, (nq / nkv) * k, at_, s));
        }

        GemmArgs go{};
        go.A = at<uint16_t>(ws, L.o);
        go.M = M;
        go.K = nq * D;
        go.W = (const uint4*)W.w_o;
        go.n_tiles = c.hidden / 16;
        go.ksteps = ks_q;
        if (io.mode == NLD_MODE_DRAFT && c.lora_rank > 0) {
            // LoRA down-projection t = lora_scale * (A o), split; the O projection then takes
            // B as lora_rank / 32 more k-steps against t
            GemmArgs gt{};
            gt.A = at<uint16_t>(ws, L.o);
            gt.M = M;
            gt.K = nq * D;
            gt.W = (const uint4*)W.lora_a;
            gt.n_tiles = c.lora_rank / 16;
            gt.ksteps = ks_q;
            gt.xg_out = at<uint16_t>(ws, L.lora_t);
            gt.out_scale = c.lora_scale;
            {
                TraceScope ts(NLD_TRACE_O_PROJ, s);
                const StreamPlan p = plan_stream(EPI_SPLIT, M, gt.n_tiles);
                HIP_TRY(launch_gemm_stream(EPI_SPLIT, p.mt, p.ct, p.nw, p.gx, p.gy, gt, s));
            }
            go.W2 = (const uint4*)W.lora_b;
            go.A2 = at<uint16_t>(ws, L.lora_t);
            go.ksteps2 = c.lora_rank / 32;
        }
        go.x = x;
        go.xg_out = at<uint16_t>(ws, L.xg);
        go.gain_next = (const uint16_t*)W.ffn_norm;
        go.part_ss_out = at<float>(ws, L.part_ss);
        go.plain = plain & SITE_NORM;
        {
            TraceScope ts(NLD_TRACE_O_PROJ, s);
            HIP_TRY(resid_gemm(SK_O, go, ws, L, s));
        }

        GemmArgs gu{};
        gu.eps = c.rms_eps;
        gu.M = M;
        gu.K = c.hidden;
        gu.W = (const uint4*)W.w_gate_up;
        gu.n_tiles = cdiv(c.ffn, 8);
        gu.ksteps = ks_h;
        gu.act = at<uint16_t>(ws, L.act);
        gu.ffn = c.ffn;
        gu.tile_ctr = at<unsigned>(ws, L.tile_ctr) + 2 * l + 1;
        gu.plain = plain & SITE_ACT;
        {
            TraceScope ts(NLD_TRACE_GATE_UP, s);
            HIP_TRY(normed_gemm(EPI_SWIGLU, gu, ws, L, s, nullptr));
        }

        GemmArgs gd{};
        gd.A = at<uint16_t>(ws, L.act);
        gd.M = M;
        gd.K = c.ffn;
        gd.W = (const uint4*)W.w_down;
        gd.n_tiles = c.hidden / 16;
        gd.ksteps = ks_f;
        gd.x = x;
        gd.xg_out = at<uint16_t>(ws, L.xg);
        gd.gain_next = (const uint16_t*)(l + 1 < c.n_layers ? mdl->layers[l + 1].attn_norm : mdl->w.final_norm);
        gd.part_ss_out = at<float>(ws, L.part_ss);
        gd.plain = plain & (l + 1 < c.n_layers ? SITE_NORM : SITE_FINAL);
        {
            TraceScope ts(NLD_TRACE_DOWN, s);
            HIP_TRY(resid_gemm(SK_DOWN, gd, ws, L, s));
        }
    }

    FinishArgs fa{};
    fa.k_blk = k;
    fa.batch = batch;
    fa.finish = io.finish;
    fa.status = status;
    fa.max_len = kv->max_len;
    fa.mask_id = c.mask_token_id;
    if (io.kv_only) {
        fa.block = io.block;
        fa.next_anchor = io.next_anchor;
        fa.lengths = kv->lengths;
        TraceScope ts(NLD_TRACE_ARGMAX, s);
        HIP_TRY(launch_finish(fa, s));
        return NLD_OK;
    }

    const bool denoise = io.finish == FINISH_DENOISE;
    const bool ensemble = io.finish == FINISH_QUAD && io.lambda > 0.0f && io.lambda < 1.0f;
    GemmArgs gl{};
    gl.tile_ctr = at<unsigned>(ws, L.tile_ctr) + 2 * c.n_layers;
    gl.eps = c.rms_eps;
    gl.M = M;
    gl.K = c.hidden;
    gl.W = (const uint4*)mdl->w.lm_head;
    gl.n_tiles = L.lm_tiles;
    gl.ksteps = ks_h;
    gl.logits = io.logits;
    gl.part_keys = at<unsigned long long>(ws, L.keys);
    gl.part_lse = (denoise || ensemble) ? at<float2>(ws, L.lse) : nullptr;
    gl.exclude_id = denoise ? c.mask_token_id : -1;
    gl.k_blk = k;
    gl.quad_k = io.quad_k;
    gl.ens_logits = ensemble ? at<float>(ws, L.ens_logits) : nullptr;
    gl.vocab = c.vocab;
    int parts = 0;
    {
        TraceScope ts(NLD_TRACE_LM_HEAD, s);
        HIP_TRY(normed_gemm(EPI_LMHEAD, gl, ws, L, s, &parts));
    }

    fa.part_keys = at<unsigned long long>(ws, L.keys);
    fa.part_lse = at<float2>(ws, L.lse);
    fa.n_parts = parts;
    fa.vocab = c.vocab;
    fa.argmax_out = io.argmax_out;
    fa.block = io.block;
    fa.threshold = io.threshold;
    fa.n_committed = io.n_committed;
    fa.n_masked = io.n_masked;
    fa.conf_out = io.conf_out;
    fa.draft_in = io.draft_in;
    fa.draft_out = io.draft_out;
    fa.accept_len = io.accept_len;
    fa.committed = io.committed;
    fa.next_anchor = io.next_anchor;
    fa.lengths = io.advance_lengths ? kv->lengths : nullptr;
    if (io.finish == FINISH_QUAD) {
        fa.quad_k = io.quad_k;
        fa.lambda = io.lambda;
        fa.ens_logits = at<float>(ws, L.ens_logits);
        fa.ens_keys = at<unsigned long long>(ws, L.ens_v);
        fa.ens_chunks = ENS_CHUNKS;
        TraceScope ts(NLD_TRACE_ARGMAX, s);
        if (ensemble) HIP_TRY(launch_quad_ensemble(fa, s));
        HIP_TRY(launch_quad_finish(fa, s));
        return NLD_OK;
    }
    {
        TraceScope ts(NLD_TRACE_ARGMAX, s);
        HIP_TRY(launch_finish(fa, s));
    }
    return NLD_OK;
}

}  // namespace

// =====================================================================================
extern "C" {

const char* nld_last_error(void) { return g_err; }

const char* nld_status_string(int32_t st) {
    switch (st) {
        case NLD_OK: return "ok";
        case NLD_ERR_INVALID_ARG: return "invalid argument";
        case NLD_ERR_SHAPE: return "unsupported shape";
        case NLD_ERR_CAPACITY: return "workspace too small";
        case NLD_ERR_HIP: return "HIP runtime error";
        case NLD_ERR_UNSUPPORTED: return "unsupported";
        case NLD_ERR_DEVICE: return "device-side error";
        default: return "unknown status";
    }
}

nld_status nld_model_create(const nld_config* cfg, const nld_weights* w, nld_model** out) {
    if (!out) return fail(NLD_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    nld_status st = check_config(cfg);
    if (st != NLD_OK) return st;
    if (!w || !w->embed || !w->final_norm || !w->lm_head || !w->layers)
        return fail(NLD_ERR_INVALID_ARG, "a model-level weight pointer is NULL");
    for (int l = 0; l < cfg->n_layers; ++l) {
        const nld_layer_weights& L = w->layers[l];
        if (!L.attn_norm || !L.w_qkv || !L.w_o || !L.ffn_norm || !L.w_gate_up || !L.w_down)
            return fail(NLD_ERR_INVALID_ARG, "a weight pointer of layer %d is NULL", l);
        if (cfg->lora_rank > 0 && (!L.lora_a || !L.lora_b))
            return fail(NLD_ERR_INVALID_ARG, "lora_rank > 0 but layer %d has no lora_a/lora_b", l);
    }
    nld_model* m = new nld_model;
    m->cfg = *cfg;
    m->w = *w;
    m->layers.assign(w->layers, w->layers + cfg->n_layers);
    m->w.layers = m->layers.data();
    *out = m;
    return NLD_OK;
}

void nld_model_destroy(nld_model* m) { delete m; }

size_t nld_packed_bytes(int32_t kind, const nld_config* cfg, int32_t out_dim, int32_t in_dim) {
    if (in_dim < 1 || out_dim < 1) return 0;
    int tiles;
    if (kind == NLD_PACK_GATE_UP) tiles = cdiv(out_dim, 8);            // out_dim = ffn
    else if (kind == NLD_PACK_QKV) {
        if (!cfg) return 0;
        tiles = (cfg->n_q_heads + 2 * cfg->n_kv_heads) * cfg->head_dim / 16;
    } else tiles = cdiv(out_dim, 16);
    return (size_t)tiles * cdiv(in_dim, 32) * 1024;
}

nld_status nld_pack_linear(const void* w, int32_t out_dim, int32_t in_dim, void* packed, void* stream) {
    if (!w || !packed) return fail(NLD_ERR_INVALID_ARG, "NULL pointer");
    if (out_dim < 1 || in_dim < 1) return fail(NLD_ERR_INVALID_ARG, "sizes must be positive");
    if (in_dim % 8) return fail(NLD_ERR_SHAPE, "in_dim (%d) must be a multiple of 8", in_dim);
    PackArgs p{};
    p.src0 = (const uint16_t*)w;
    p.kind = PACK_LINEAR;
    p.out_dim = out_dim;
    p.in_dim = in_dim;
    p.n_tiles = cdiv(out_dim, 16);
    p.ksteps = cdiv(in_dim, 32);
    p.dst = (uint4*)packed;
    HIP_TRY(launch_pack(p, (hipStream_t)stream));
    return NLD_OK;
}

nld_status nld_pack_qkv(const nld_config* cfg, const void* wq, const void* wk, const void* wv, void* packed,
                        void* stream) {
    nld_status st = check_config(cfg);
    if (st != NLD_OK) return st;
    if (!wq || !wk || !wv || !packed) return fail(NLD_ERR_INVALID_ARG, "NULL pointer");
    PackArgs p{};
    p.src0 = (const uint16_t*)wq;
    p.src1 = (const uint16_t*)wk;
    p.src2 = (const uint16_t*)wv;
    p.kind = PACK_QKV;
    p.head_dim = cfg->head_dim;
    p.rows0 = cfg->n_q_heads * cfg->head_dim;
    p.rows1 = cfg->n_kv_heads * cfg->head_dim;
    p.out_dim = p.rows0 + 2 * p.rows1;
    p.in_dim = cfg->hidden;
    p.n_tiles = p.out_dim / 16;
    p.ksteps = cdiv(cfg->hidden, 32);
    p.dst = (uint4*)packed;
    HIP_TRY(launch_pack(p, (hipStream_t)stream));
    return NLD_OK;
}

nld_status nld_pack_gate_up(const nld_config* cfg, const void* wg, const void* wu, void* packed, void* stream) {
    nld_status st = check_config(cfg);
    if (st != NLD_OK) return st;
    if (!wg || !wu || !packed) return fail(NLD_ERR_INVALID_ARG, "NULL pointer");
    PackArgs p{};
    p.src0 = (const uint16_t*)wg;
    p.src1 = (const uint16_t*)wu;
    p.kind = PACK_GATE_UP;
    p.rows0 = cfg->ffn;
    p.out_dim = 2 * cfg->ffn;
    p.in_dim = cfg->hidden;
    p.n_tiles = cdiv(cfg->ffn, 8);
    p.ksteps = cdiv(cfg->hidden, 32);
    p.dst = (uint4*)packed;
    HIP_TRY(launch_pack(p, (hipStream_t)stream));
    return NLD_OK;
}

size_t nld_workspace_bytes(const nld_model* m, int32_t batch, int32_t k, int32_t max_len) {
    if (!m || batch < 1 || k < 1 || max_len < 64) return 0;
    return make_layout(m->cfg, batch, k, max_len).total;
}

nld_status nld_workspace_init(void* workspace, size_t ws_bytes, void* stream) {
    if (!workspace) return fail(NLD_ERR_INVALID_ARG, "workspace is NULL");
    if (ws_bytes < 256) return fail(NLD_ERR_CAPACITY, "workspace too small");
    HIP_TRY(launch_fill_zero(workspace, ws_bytes & ~(size_t)3, (hipStream_t)stream));
    return NLD_OK;
}

nld_status nld_block_forward(const nld_model* m, const nld_kv_cache* kv, const int32_t* tokens, int32_t batch,
                             int32_t k, int32_t mode, int32_t bidir_from, float* logits, int32_t* argmax,
                             void* workspace, size_t ws_bytes, void* stream) {
    Layout L;
    nld_status st = validate_call(m, kv, batch, k, workspace, ws_bytes, &L);
    if (st != NLD_OK) return st;
    if (!tokens) return fail(NLD_ERR_INVALID_ARG, "tokens is NULL");
    if (mode != NLD_MODE_VERIFY && mode != NLD_MODE_DRAFT) return fail(NLD_ERR_INVALID_ARG, "mode must be 0 or 1");
    if (bidir_from < 0 || bidir_from > k) return fail(NLD_ERR_INVALID_ARG, "bidir_from must be in [0, k]");
    PassIO io{};
    io.source = SRC_TOKENS;
    io.tokens = tokens;
    io.mode = mode;
    io.bidir_from = bidir_from;
    io.logits = logits;
    io.argmax_out = argmax;
    io.finish = FINISH_NONE;
    return run_pass(m, kv, batch, k, io, workspace, L, (hipStream_t)stream);
}

nld_status nld_draft(const nld_model* m, const nld_kv_cache* kv, const int32_t* anchor, int32_t batch, int32_t k,
                     int32_t bidir_from, int32_t* draft, float* logits, void* workspace, size_t ws_bytes,
                     void* stream) {
    Layout L;
    nld_status st = validate_call(m, kv, batch, k, workspace, ws_bytes, &L);
    if (st != NLD_OK) return st;
    if (k < 2) return fail(NLD_ERR_INVALID_ARG, "a draft needs k >= 2");
    if (!anchor || !draft) return fail(NLD_ERR_INVALID_ARG, "anchor or draft is NULL");
    if (bidir_from < 0 || bidir_from > k) return fail(NLD_ERR_INVALID_ARG, "bidir_from must be in [0, k]");
    PassIO io{};
    io.source = SRC_DRAFT;
    io.anchor = anchor;
    io.mode = NLD_MODE_DRAFT;
    io.bidir_from = bidir_from;
    io.logits = logits;
    io.finish = FINISH_DRAFT;
    io.draft_out = draft;
    return run_pass(m, kv, batch, k, io, workspace, L, (hipStream_t)stream);
}

nld_status nld_verify_accept(const nld_model* m, const nld_kv_cache* kv, const int32_t* anchor,
                             const int32_t* draft, int32_t batch, int32_t k, int32_t* accept_len,
                             int32_t* committed, int32_t* next_anchor, float* logits, void* workspace,
                             size_t ws_bytes, void* stream) {
    Layout L;
    nld_status st = validate_call(m, kv, batch, k, workspace, ws_bytes, &L);
    if (st != NLD_OK) return st;
    if (!anchor || !accept_len || !committed || !next_anchor)
        return fail(NLD_ERR_INVALID_ARG, "anchor, accept_len, committed or next_anchor is NULL");
    if (k > 1 && !draft) return fail(NLD_ERR_INVALID_ARG, "draft is NULL");
    PassIO io{};
    io.source = SRC_VERIFY;
    io.anchor = anchor;
    io.draft_in = draft;
    io.mode = NLD_MODE_VERIFY;
    io.logits = logits;
    io.finish = FINISH_ACCEPT;
    io.accept_len = accept_len;
    io.committed = committed;
    io.next_anchor = next_anchor;
    io.advance_lengths = true;
    return run_pass(m, kv, batch, k, io, workspace, L, (hipStream_t)stream);
}

size_t nld_quad_workspace_bytes(const nld_model* m, int32_t batch, int32_t k, int32_t max_len) {
    if (!m || batch < 1 || k < 2 || k > NLD_QUAD_MAX_K || max_len < 1) return 0;
    return make_layout(m->cfg, batch, k * (k + 1), max_len, k).total;
}

nld_status nld_quad_step(const nld_model* m, const nld_kv_cache* kv, const int32_t* anchor, const int32_t* spec,
                         int32_t batch, int32_t k, float lambda, int32_t* accept_len, int32_t* committed,
                         int32_t* next_anchor, int32_t* next_spec, float* logits, void* workspace, size_t ws_bytes,
                         void* stream) {
    if (k < 2 || k > NLD_QUAD_MAX_K) return fail(NLD_ERR_INVALID_ARG, "quadratic k must be in [2, %d] (got %d)",
                                                 NLD_QUAD_MAX_K, k);
    if (!(lambda >= 0.0f && lambda <= 1.0f)) return fail(NLD_ERR_INVALID_ARG, "lambda must be in [0, 1]");
    Layout L;
    nld_status st = validate_call(m, kv, batch, k * (k + 1), workspace, ws_bytes, &L, k);
    if (st != NLD_OK) return st;
    if (!anchor || !spec || !accept_len || !committed || !next_anchor || !next_spec)
        return fail(NLD_ERR_INVALID_ARG, "anchor, spec, accept_len, committed, next_anchor or next_spec is NULL");
    PassIO io{};
    io.source = SRC_QUAD;
    io.anchor = anchor;
    io.draft_in = spec;
    io.mode = NLD_MODE_QUAD_INTERNAL;
    io.logits = logits;
    io.finish = FINISH_QUAD;
    io.accept_len = accept_len;
    io.committed = committed;
    io.next_anchor = next_anchor;
    io.draft_out = next_spec;
    io.advance_lengths = true;
    io.quad_k = k;
    io.lambda = lambda;
    return run_pass(m, kv, batch, k * (k + 1), io, workspace, L, (hipStream_t)stream);
}

nld_status nld_denoise_step(const nld_model* m, const nld_kv_cache* kv, int32_t* block, int32_t batch, int32_t k,
                            int32_t bidir_from, float threshold, int32_t* n_committed, int32_t* n_masked,
                            float* confidence, float* logits, void* workspace, size_t ws_bytes, void* stream) {
    Layout L;
    nld_status st = validate_call(m, kv, batch, k, workspace, ws_bytes, &L);
    if (st != NLD_OK) return st;
    if (k < 2) return fail(NLD_ERR_INVALID_ARG, "a denoising step needs k >= 2");
    if (m->cfg.vocab < 2) return fail(NLD_ERR_SHAPE, "denoising needs a vocabulary besides the mask token");
    if (!block || !n_committed || !n_masked) return fail(NLD_ERR_INVALID_ARG, "block, n_committed or n_masked is NULL");
    if (bidir_from < 0 || bidir_from > k) return fail(NLD_ERR_INVALID_ARG, "bidir_from must be in [0, k]");
    if (threshold != threshold) return fail(NLD_ERR_INVALID_ARG, "threshold is NaN");
    PassIO io{};
    io.source = SRC_TOKENS;
    io.tokens = block;
    io.mode = NLD_MODE_DRAFT;
    io.bidir_from = bidir_from;
    io.logits = logits;
    io.finish = FINISH_DENOISE;
    io.block = block;
    io.threshold = threshold;
    io.n_committed = n_committed;
    io.n_masked = n_masked;
    io.conf_out = confidence;
    return run_pass(m, kv, batch, k, io, workspace, L, (hipStream_t)stream);
}

nld_status nld_refresh_block(const nld_model* m, const nld_kv_cache* kv, const int32_t* block, int32_t batch,
                             int32_t k, int32_t* next_anchor, void* workspace, size_t ws_bytes, void* stream) {
    Layout L;
    nld_status st = validate_call(m, kv, batch, k, workspace, ws_bytes, &L);
    if (st != NLD_OK) return st;
    if (k < 2) return fail(NLD_ERR_INVALID_ARG, "a refresh needs k >= 2");
    if (!block || !next_anchor) return fail(NLD_ERR_INVALID_ARG, "block or next_anchor is NULL");
    PassIO io{};
    io.source = SRC_TOKENS;
    io.tokens = block;
    io.mode = NLD_MODE_VERIFY;
    io.finish = FINISH_REFRESH;
    io.block = (int32_t*)block;   // read only
    io.next_anchor = next_anchor;
    io.kv_only = true;
    return run_pass(m, kv, batch, k, io, workspace, L, (hipStream_t)stream);
}

nld_status nld_commit_from_logits(const float* logits, int32_t* block, int32_t batch, int32_t k, int32_t vocab,
                                  int32_t mask_token_id, float threshold, int32_t* argmax, int32_t* n_committed,
                                  int32_t* n_masked, float* confidence, void* stream) {
    if (!logits || !block || !n_committed || !n_masked) return fail(NLD_ERR_INVALID_ARG, "NULL pointer");
    if (batch < 1 || k < 2 || k > 64 || vocab < 2) return fail(NLD_ERR_INVALID_ARG, "bad batch, k or vocab");
    if (mask_token_id < 0 || mask_token_id >= vocab) return fail(NLD_ERR_INVALID_ARG, "mask_token_id outside [0, vocab)");
    if (threshold != threshold) return fail(NLD_ERR_INVALID_ARG, "threshold is NaN");
    FinishArgs fa{};
    fa.logits = logits;
    fa.vocab = vocab;
    fa.k_blk = k;
    fa.batch = batch;
    fa.argmax_out = argmax;
    fa.finish = FINISH_DENOISE;
    fa.block = block;
    fa.mask_id = mask_token_id;
    fa.threshold = threshold;
    fa.n_committed = n_committed;
    fa.n_masked = n_masked;
    fa.conf_out = confidence;
    HIP_TRY(launch_finish(fa, (hipStream_t)stream));
    return NLD_OK;
}

nld_status nld_decode_steps(const nld_model* m, const nld_kv_cache* kv, int32_t* anchor, int32_t batch, int32_t k,
                            int32_t n_steps, int32_t bidir_from, int32_t* accept_len, int32_t* committed,
                            void* workspace, size_t ws_bytes, void* stream) {
    Layout L;
    nld_status st = validate_call(m, kv, batch, k, workspace, ws_bytes, &L);
    if (st != NLD_OK) return st;
    if (n_steps < 1) return fail(NLD_ERR_INVALID_ARG, "n_steps must be >= 1");
    if (!anchor || !accept_len || !committed) return fail(NLD_ERR_INVALID_ARG, "anchor, accept_len or committed is NULL");
    if (bidir_from < 0 || bidir_from > k) return fail(NLD_ERR_INVALID_ARG, "bidir_from must be in [0, k]");
    int32_t* drafts = at<int32_t>(workspace, L.drafts);
    hipStream_t s = (hipStream_t)stream;
    for (int step = 0; step < n_steps; ++step) {
        if (k >= 2) {
            PassIO d{};
            d.source = SRC_DRAFT;
            d.anchor = anchor;
            d.mode = NLD_MODE_DRAFT;
            d.bidir_from = bidir_from;
            d.finish = FINISH_DRAFT;
            d.draft_out = drafts;
            st = run_pass(m, kv, batch, k, d, workspace, L, s);
            if (st != NLD_OK) return st;
        }
        PassIO v{};
        v.source = SRC_VERIFY;
        v.anchor = anchor;
        v.draft_in = drafts;
        v.mode = NLD_MODE_VERIFY;
        v.finish = FINISH_ACCEPT;
        v.accept_len = accept_len + (size_t)step * batch;
        v.committed = committed + (size_t)step * batch * k;
        v.next_anchor = anchor;   // written last by the finish kernel: the next step's anchor
        v.advance_lengths = true;
        st = run_pass(m, kv, batch, k, v, workspace, L, s);
        if (st != NLD_OK) return st;
    }
    return NLD_OK;
}

int32_t nld_choose_block(float ar_step_ms, float ss_step_ms, float expected_committed, int32_t k_ss) {
    if (!(ar_step_ms > 0.f) || !(ss_step_ms > 0.f) || k_ss < 2) return 1;
    // committed tokens per millisecond: 1 per AR step, expected_committed per self-speculation step
    return expected_committed / ss_step_ms > 1.0f / ar_step_ms ? k_ss : 1;
}

size_t nld_accept_workspace_bytes(int32_t batch, int32_t k) {
    if (batch < 1 || k < 1) return 0;
    return 256;
}

nld_status nld_accept_from_logits(const float* logits, const int32_t* draft, int32_t batch, int32_t k,
                                  int32_t vocab, int32_t* argmax, int32_t* accept_len, int32_t* committed,
                                  int32_t* next_anchor, void* workspace, size_t ws_bytes, void* stream) {
    if (!logits || !argmax || !accept_len || !committed || !next_anchor || !workspace)
        return fail(NLD_ERR_INVALID_ARG, "NULL pointer");
    if (batch < 1 || k < 1 || k > 64 || vocab < 1) return fail(NLD_ERR_INVALID_ARG, "bad batch, k or vocab");
    if (k > 1 && !draft) return fail(NLD_ERR_INVALID_ARG, "draft is NULL");
    if (ws_bytes < nld_accept_workspace_bytes(batch, k)) return fail(NLD_ERR_CAPACITY, "workspace too small");
    FinishArgs fa{};
    fa.part_keys = nullptr;
    fa.logits = logits;
    fa.vocab = vocab;
    fa.k_blk = k;
    fa.batch = batch;
    fa.argmax_out = argmax;
    fa.finish = FINISH_ACCEPT;
    fa.draft_in = draft;
    fa.accept_len = accept_len;
    fa.committed = committed;
    fa.next_anchor = next_anchor;
    HIP_TRY(launch_finish(fa, (hipStream_t)stream));
    return NLD_OK;
}

nld_status nld_trace_enable(int32_t on) {
    g_trace_on = on != 0;
    return NLD_OK;
}

nld_status nld_trace_read(float* ms, int32_t* counts, int32_t n) {
    if (!ms || !counts || n < NLD_TRACE_CLASSES) return fail(NLD_ERR_INVALID_ARG, "need host arrays of NLD_TRACE_CLASSES");
    for (int i = 0; i < n; ++i) {
        ms[i] = 0.f;
        counts[i] = 0;
    }
    nld_status st = NLD_OK;
    for (TraceRec& r : g_trace) {
        float t = 0.f;
        if (st == NLD_OK) {
            hipError_t e = hipEventSynchronize(r.stop);
            if (e == hipSuccess) e = hipEventElapsedTime(&t, r.start, r.stop);
            if (e != hipSuccess) st = fail(NLD_ERR_HIP, "trace event: %s", hipGetErrorString(e));
        }
        ms[r.cls] += t;
        counts[r.cls] += r.first ? 1 : 0;
        (void)hipEventDestroy(r.start);
        (void)hipEventDestroy(r.stop);
    }
    g_trace.clear();
    return st;
}

nld_status nld_read_device_status(void* workspace, uint32_t* host_bits, void* stream) {
    if (!workspace || !host_bits) return fail(NLD_ERR_INVALID_ARG, "NULL pointer");
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(hipStreamSynchronize(s));
    HIP_TRY(hipMemcpy(host_bits, workspace, 4, hipMemcpyDeviceToHost));
    HIP_TRY(launch_fill_zero(workspace, 4, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (*host_bits) return fail(NLD_ERR_DEVICE, "device status bits 0x%x", *host_bits);
    return NLD_OK;
}

}  // extern "C"

// ---------------------------------------------------------------- allocation-free verify
// The scratch of nld_verify_accept_noalloc: one copy per device, loaded with the code object.  In host
// code `scratch` is a stand-in symbol, not a device address; the address each device's copy has comes
// from hipGetSymbolAddress (with that device current) and is kept per device.  Only that address is
// ever passed to a kernel or a fill.
static __device__ __align__(256) unsigned char scratch[NLD_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

// This device's scratch address; on the device's first call the whole array is zeroed (a fill kernel on
// `s`), which is the state nld_workspace_init gives a workspace.
nld_status scratch_of_current_device(hipStream_t s, void** out) {
    int dev = -1;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= MAX_DEVICES) return fail(NLD_ERR_UNSUPPORTED, "device ordinal %d outside [0, %d)", dev, MAX_DEVICES);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return fail(NLD_ERR_HIP, "hipGetSymbolAddress gave no address for the scratch array");
        HIP_TRY(launch_fill_zero(p, NLD_NOALLOC_SCRATCH_BYTES, s));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return NLD_OK;
}

}  // namespace

extern "C" {

nld_status nld_verify_accept_noalloc(const nld_model* m, const nld_kv_cache* kv, const int32_t* anchor,
                                     const int32_t* draft, int32_t batch, int32_t k, int32_t* accept_len,
                                     int32_t* committed, int32_t* next_anchor, float* logits,
                                     uint32_t* device_status, void* stream) {
    // host checks first, with a non-null stand-in workspace of the maximal size: the layout of this call
    // must fit the scratch array before anything touches the device
    Layout L;
    nld_status st = validate_call(m, kv, batch, k, (void*)&g_scratch_mu, NLD_NOALLOC_SCRATCH_BYTES, &L);
    if (st == NLD_ERR_CAPACITY)
        return fail(NLD_ERR_CAPACITY, "this batch (%d), k (%d) and max_len (%d) need %zu bytes of scratch; the "
                    "allocation-free entry point holds at most %u", batch, k, kv->max_len, L.total,
                    (unsigned)NLD_NOALLOC_SCRATCH_BYTES);
    if (st != NLD_OK) return st;
    if (!anchor || !accept_len || !committed || !next_anchor)
        return fail(NLD_ERR_INVALID_ARG, "anchor, accept_len, committed or next_anchor is NULL");
    if (k > 1 && !draft) return fail(NLD_ERR_INVALID_ARG, "draft is NULL");
    hipStream_t s = (hipStream_t)stream;
    void* ws = nullptr;
    st = scratch_of_current_device(s, &ws);
    if (st != NLD_OK) return st;
    uint32_t* status = at<uint32_t>(ws, L.status);
    HIP_TRY(launch_fill_zero(status, 4, s));
    PassIO io{};
    io.source = SRC_VERIFY;
    io.anchor = anchor;
    io.draft_in = draft;
    io.mode = NLD_MODE_VERIFY;
    io.logits = logits;
    io.finish = FINISH_ACCEPT;
    io.accept_len = accept_len;
    io.committed = committed;
    io.next_anchor = next_anchor;
    io.advance_lengths = true;
    st = run_pass(m, kv, batch, k, io, ws, L, s);
    if (st != NLD_OK) return st;
    if (device_status) HIP_TRY(launch_copy_u32(status, device_status, s));
    return NLD_OK;
}

}  // extern "C"
