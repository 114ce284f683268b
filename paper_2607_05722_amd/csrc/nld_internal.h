// Internal declarations shared by the kernels and the host API of libnld.
// gfx950 (CDNA4) only: 64-wide wavefronts, v_mfma_f32_16x16x32_bf16.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace nld {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

// ---------------------------------------------------------------- numerics helpers
__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// float -> bfloat16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950)
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f);
}
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
// two floats -> packed bfloat16 pair (lo in bits 0..15), one conversion instruction
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// C[16x16] += A[16x32] * B[32x16].  Lane l supplies A[l%16][8(l/16)..+8] and
// B[8(l/16)..+8][l%16] (8 bf16 each, one 16-byte register quad) and holds
// C[4(l/16)+i][l%16], i = 0..3.
__device__ __forceinline__ f32x4_t mfma_16x16x32(uint4 a, uint4 b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
}

// One 16-byte block of a weight matrix that is read once per pass, loaded with the non-temporal
// hint (the `nt` bit).  The normed GEMMs use it for their weight streams, where it measured
// faster; the O, down and attention streams measured slower with it and keep plain loads.
__device__ __forceinline__ uint4 load_stream(const uint4* p) {
    typedef uint32_t u32x4_nt __attribute__((ext_vector_type(4)));
    const u32x4_nt v = __builtin_nontemporal_load((const u32x4_nt*)p);
    return uint4{v[0], v[1], v[2], v[3]};
}

// Order-preserving key for a float value at column n: larger value wins, then
// lower column.  -0.0 is folded onto +0.0 so that equal values tie on index.
__device__ __forceinline__ unsigned long long argmax_key(float v, uint32_t n) {
    uint32_t u = __float_as_uint(v);
    if ((u & 0x7FFFFFFFu) == 0u) u = 0u;
    uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((unsigned long long)ord << 32) | (unsigned long long)(0xFFFFFFFFu - n);
}
__device__ __forceinline__ int32_t argmax_key_index(unsigned long long key) {
    return (int32_t)(0xFFFFFFFFu - (uint32_t)(key & 0xFFFFFFFFull));
}

// Activation operands (the A side of every projection) are split and stored in
// MFMA operand order.  Split: a value a is carried as two bfloat16 numbers,
// hi = bf16(a) and lo = bf16(a - hi); against an exact bf16 weight, hi*w + lo*w
// (two MFMAs, fp32 accumulation) keeps about 16 significant bits of a instead of
// 8.  Operand order: rows in tiles of 16, columns in steps of 32; tile mt, step s
// is a 1 KiB hi block whose 16-byte lane l holds A[16mt + l%16][32s + 8(l/16) .. +8],
// followed by the lo block of the same shape, so a wavefront fetches each half
// of an operand with one contiguous 1 KiB load.  Returns the index of the hi value.
__host__ __device__ __forceinline__ size_t split_index(int m, int k, int ksteps) {
    return ((size_t)(((m >> 4) * ksteps + (k >> 5)) * 2) * 64 + (size_t)((((k & 31) >> 3) << 4) + (m & 15))) * 8 + (k & 7);
}
constexpr int SPLIT_LO = 512;   // element offset of a lo value from its hi value

// plain != 0: the operand site is carried in plain bf16 (the lo value is stored as zero)
__device__ __forceinline__ void store_split(uint16_t* p, size_t hi_index, float v, int plain = 0) {
    const uint32_t h = f32_to_bf16(v);
    p[hi_index] = (uint16_t)h;
    p[hi_index + SPLIT_LO] = plain ? (uint16_t)0 : (uint16_t)f32_to_bf16(v - bf16_to_f32(h));
}

// eight floats -> hi and lo operand quads (element e in bits 16(e%2) of word e/2); plain: lo = 0
__device__ __forceinline__ void split8(const float* v, uint4& hi, uint4& lo, int plain = 0) {
    uint32_t h[4], l[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        h[q] = pack_bf16x2(v[2 * q], v[2 * q + 1]);
        l[q] = pack_bf16x2(v[2 * q] - bf16_to_f32(h[q] & 0xFFFFu), v[2 * q + 1] - bf16_to_f32(h[q] >> 16));
    }
    hi = uint4{h[0], h[1], h[2], h[3]};
    lo = plain ? uint4{0u, 0u, 0u, 0u} : uint4{l[0], l[1], l[2], l[3]};
}

// Operand sites that may be carried in plain bf16 instead of split (hi + lo) form: a precision
// knob (NLD_PLAIN_SITES on the host); every site is split by default.
enum PlainSite : uint32_t {
    SITE_NORM = 1u,    // RMSNorm operands of the QKV and gate/up projections
    SITE_FINAL = 2u,   // the final RMSNorm operand (LM head input)
    SITE_Q = 4u,       // queries
    SITE_KV = 8u,      // the block's own keys and values (the attention's in-pass copy)
    SITE_P = 16u,      // attention probabilities
    SITE_O = 32u,      // attention output (O projection input)
    SITE_ACT = 64u     // SwiGLU output (down projection input)
};

// ---------------------------------------------------------------- kernel arguments
enum EpiKind { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LMHEAD = 3, EPI_SPLIT = 4 };

struct GemmArgs {
    // A operand: split bf16 activations in operand order (split_index with `ksteps`).
    // For the projections whose input is RMSNorm(x) (QKV, gate/up, LM head) A is
    // x * gain, written by the kernel that produced x, and part_ss holds that
    // producer's sums of x^2 over 16-column chunks ([M][n_ss]); the consumer turns
    // them into 1/rms per row.
    const uint16_t* A;
    const float* part_ss;
    int n_ss;
    float eps;
    int M;               // rows
    int K;               // reduction length (multiple of 8)
    const uint4* W;      // packed weights: [n_tiles][ksteps][64 lanes] x 16 bytes
    int n_tiles;
    int ksteps;          // ceil(K / 32)
    unsigned* tile_ctr;  // normed GEMM: dynamic tile counter (zeroed by the embedding kernel each pass)
    // Second reduction source (streamed GEMM only, ksteps2 <= 2 * wavefronts): the sum
    // continues over ksteps2 more k-steps of W2 (packed, ksteps2 steps per tile) against A2
    // (split, ksteps2 steps per row tile).  The draft pass's O projection uses it for the
    // LoRA up-projection.
    const uint4* W2;
    const uint16_t* A2;
    int ksteps2;
    // EPI_SPLIT: xg_out gets the split operand out_scale * (A W^T) (split_index with n_tiles/2 steps)
    float out_scale;
    // EPI_RESID: x += A W^T, then the next RMSNorm's operand and statistics
    float* x;
    uint16_t* xg_out;          // split x * gain_next, split_index with N/32 steps
    const uint16_t* gain_next;
    float* part_ss_out;        // [M][N/16]
    // EPI_QKV
    uint16_t* q_out;     // split bf16 queries in the attention's operand order (q_index)
    int q_row_tiles;     // query-row tiles of 16 per (sequence, KV head)
    uint16_t* kc;        // this layer's K cache [batch][n_kv_heads][max_len][head_dim]
    uint16_t* vc;        // this layer's V cache [batch][n_kv_heads][max_len/64][head_dim][64]
    int write_cache;     // verify: the block's K/V rows also go to cache rows [P_b, P_b + k)
    uint16_t* blk_k;     // the block's own keys, split: [unit][hi, lo][64 rows][head_dim]
    uint16_t* blk_v;     // the block's own values, split: [unit][hi, lo][head_dim][64 rows]
    const int32_t* lengths;
    int k_blk;
    int n_q_heads, n_kv_heads, head_dim, max_len;
    const float2* rope;  // [M][head_dim/2] (cos, sin) of each row's RoPE angles (embedding kernel)
    uint32_t* status;
    // EPI_SWIGLU
    uint16_t* act;       // split bf16 silu(gate) * up, split_index with ceil(ffn/32) steps
    int ffn;
    // EPI_LMHEAD
    float* logits;                   // optional f32 [M][vocab]
    unsigned long long* part_keys;   // [M][n_parts]: one argmax key per row per workgroup
    float2* part_lse;                // optional [M][n_parts]: (max, sum of exp(z - max)) per row per workgroup
    int exclude_id;                  // column left out of the argmax and the sums (-1: none)
    int n_parts;
    int vocab;
    // Quadratic self-speculation: quad_k chain rows lead every block of k_blk = quad_k * (quad_k + 1)
    // rows (then quad_k groups of quad_k masks).  Only chain rows write the cache; the LM head
    // copies the logits of the verifier rows (chain row i and mask 1 of group i, i < quad_k) to
    // ens_logits [batch][2 * quad_k][vocab] when that buffer is given.
    int quad_k;
    float* ens_logits;
    // PlainSite bits of the split operands this GEMM's epilogue writes (EPI_QKV: SITE_Q and SITE_KV;
    // EPI_SWIGLU: SITE_ACT; EPI_RESID: SITE_NORM, or SITE_FINAL when gain_next is the final norm's)
    uint32_t plain;
};

// Queries are stored per (sequence b, KV head) unit with the unit's rows
// (row = local head * k + block row j) in tiles of 16 and head dims in steps of
// 32, in MFMA operand order, split: one 1 KiB hi block and its 1 KiB lo block per
// (row tile, step).  Returns the index of the hi value.
__host__ __device__ __forceinline__ size_t q_index(int unit, int row, int d, int row_tiles, int D) {
    return ((size_t)(((unit * row_tiles + (row >> 4)) * (D >> 5) + (d >> 5)) * 2) * 64 + (size_t)((((d & 31) >> 3) << 4) + (row & 15))) * 8 + (d & 7);
}

struct AttnArgs {
    const uint16_t* q;   // split bf16 queries (q_index)
    const uint16_t* kc;  // this layer's K cache
    const uint16_t* vc;  // this layer's V cache (64-position transposed tiles)
    const uint16_t* blk_k;  // the block's keys and values in split form (GemmArgs::blk_k, blk_v)
    const uint16_t* blk_v;
    const int32_t* lengths;
    uint16_t* o;         // split bf16 attention output, split_index with n_q_heads*D/32 steps
    float* part_o;       // [units][n_parts][rows_pad][D]
    float* part_ml;      // [units][n_parts][rows_pad][2]
    int k_blk, n_q_heads, n_kv_heads, max_len, n_splits, chunk, mode, bidir_from, rows_pad;
    int row_tiles;       // query-row tiles of 16 per unit (GQA group size x k / 16, rounded up)
    int quad_k;          // mode 2 (quadratic self-speculation): chain length of the block's layout
    int n_parts;         // partial results per (unit, row): n_splits prefix splits + the block part
    float scale_log2;    // log2(e) / sqrt(D)
    // Length-aware work (batches): grid.x counts (unit, split) items numbered unit by unit from the
    // committed lengths, unit u of sequence b taking ceil(P_b / chunk) prefix splits and the block
    // part; items past the total leave at once, and the merge reads only the valid parts.
    int items;
    int n_seq;           // sequences (units / n_kv_heads)
    uint32_t plain;      // PlainSite bits: SITE_P (probabilities), SITE_O (the merged output)
    int late;            // prefix stages 1, 2 requested: 0 with the first, 1 stage 2 once the first is in
                         // LDS, 2 both once the first is in LDS
};

struct EmbedArgs {
    const int32_t* tokens;  // source 0: [batch][k]
    const int32_t* anchor;  // sources 1, 2: [batch]
    const int32_t* draft;   // source 2: [batch][k-1]
    int source;             // 0 tokens, 1 draft block, 2 verify block
    int k_blk, M, mask_id, vocab, hidden;
    const uint16_t* embed;
    const uint16_t* gain;   // first layer's attention RMSNorm gain
    float* x;
    uint16_t* xg;           // split x * gain, split_index with hidden/32 steps
    float* part_ss;         // [M][hidden/16]
    uint32_t* status;
    unsigned* tile_ctr;     // [n_tile_ctr] dynamic tile counters of this pass's GEMMs, zeroed here
    int n_tile_ctr;
    // RoPE table: rope[m][i] = (cos, sin) of (P_b + j) * inv_freq[i], i < head_dim/2
    float2* rope;
    const int32_t* lengths;
    int max_len, head_dim;
    int quad_k;             // source 3: chain length of the quadratic layout (block row positions follow it)
    uint32_t plain;         // SITE_NORM: the first layer's RMSNorm operand in plain bf16
    double inv_freq[64];    // base^(-2i/head_dim), computed on the host in fp64
};

enum FinishKind {
    FINISH_NONE = 0, FINISH_DRAFT = 1, FINISH_ACCEPT = 2, FINISH_DENOISE = 3, FINISH_REFRESH = 4, FINISH_QUAD = 5
};

struct FinishArgs {
    const unsigned long long* part_keys;  // [M][n_parts] (or NULL: reduce `logits`)
    int n_parts;
    const float* logits;                  // [M][vocab]
    int vocab;
    int k_blk, batch;
    int32_t* argmax_out;                  // optional [M]
    int finish;
    const int32_t* draft_in;              // FINISH_ACCEPT: [batch][k-1]
    int32_t* draft_out;                   // FINISH_DRAFT: [batch][k-1]
    int32_t* accept_len;
    int32_t* committed;                   // [batch][k]
    int32_t* next_anchor;
    int32_t* lengths;                     // advanced by L+1 (may be NULL); FINISH_REFRESH: by k-1
    int max_len;                          // cache capacity: a length never advances past it (DEV_CAPACITY)
    // FINISH_DENOISE: confidence-threshold commit into `block`; FINISH_REFRESH: reads `block`
    const float2* part_lse;               // [M][n_parts] (NULL with `logits`: reduced from them)
    int32_t* block;                       // [batch][k]
    int mask_id;                          // left out of the denoising argmax and softmax
    float threshold;
    int32_t* n_committed;                 // [batch]
    int32_t* n_masked;                    // [batch] masks left after the commit
    float* conf_out;                      // optional [M]
    uint32_t* status;
    // FINISH_QUAD: chain length quad_k (k_blk = quad_k * (quad_k + 1) rows per sequence); draft_in
    // holds the speculative tokens [batch][quad_k - 1], draft_out receives the next ones; the
    // verifier is the AR row (lambda >= 1), the diffusion row (lambda <= 0) or, in between, the
    // ensemble kernel's argmax keys ens_keys [batch][quad_k][ens_chunks] (one per vocabulary
    // chunk, from ens_logits and part_lse).
    int quad_k;
    float lambda;
    const float* ens_logits;
    unsigned long long* ens_keys;
    int ens_chunks;
};

enum PackKind { PACK_LINEAR = 0, PACK_QKV = 1, PACK_GATE_UP = 2 };

struct PackArgs {
    const uint16_t* src0;
    const uint16_t* src1;
    const uint16_t* src2;
    int kind;
    int out_dim, in_dim, n_tiles, ksteps;
    int head_dim, rows0, rows1;  // QKV: rows of wq and wk; GATE_UP: ffn in rows0
    uint4* dst;
};

// ---------------------------------------------------------------- launch tracing (api.hip)
// While tracing is on, returns true with a fresh pair of events for the next launch, which
// then records them on its own dispatch (start and end of the kernel itself).
bool trace_launch_events(hipEvent_t* start, hipEvent_t* stop);

// ---------------------------------------------------------------- launchers (kernels.hip)
hipError_t launch_pack(const PackArgs& a, hipStream_t s);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);
hipError_t launch_copy_u32(const uint32_t* src, uint32_t* dst, hipStream_t s);   // *dst = *src (one word)
hipError_t launch_embed(const EmbedArgs& a, hipStream_t s);
// Normed multi-tile GEMM (M <= 16).  ks = k-steps per wavefront (ksteps = ks * waves); grid = workgroups.
bool gemm_norm_supported(int ks);
int gemm_norm_max_waves(int ks);
hipError_t launch_gemm_norm(int epi, int ks, int waves, int grid, const GemmArgs& a, hipStream_t s);
// Streamed GEMM: 16*mt rows x 16*ct columns per workgroup, nw wavefronts split K.
// normed: the operand is an RMSNorm output (per-row scale from part_ss).
// With a.W2 set (EPI_RESID only) the reduction continues over the second source.
hipError_t launch_gemm_stream(int epi, int mt, int ct, int nw, int grid_x, int grid_y, const GemmArgs& a,
                              hipStream_t s);
// Normed multi-tile GEMM for 17..64 rows (EPI_QKV, EPI_SWIGLU, EPI_LMHEAD) with the K split
// into slices of gemm_normk_kstep_span(M) k-steps (grid grid_x x slices); the slices meet in
// `part` (n_tiles * slices * 256 * MT floats) through one counter per column tile in `tctr`
// (zero before the launch and zero again after it).  LM head: n_parts = grid_x * slices.
// Needs ceil(n_tiles / grid_x) <= gemm_normk_max_tiles().
bool gemm_normk_supported(int epi, int M);
int gemm_normk_kstep_span(int M);
int gemm_normk_max_tiles();
hipError_t launch_gemm_normk(int epi, int grid_x, const GemmArgs& a, float* part, unsigned* tctr, hipStream_t s);
// Split-K GEMM (EPI_RESID, EPI_QKV or EPI_SWIGLU; M <= 64, no second source): ct column
// tiles per workgroup (2..4), the reduction cut into ksplit slices (1..SPLITK_MAX) whose
// partials meet in `part` (ceil(n_tiles/ct) * ksplit * 256*ct*MT floats, MT = 1, 2 or 4 row
// tiles for M <= 16, 32, 64; unused with ksplit = 1); `ctr`
// holds one counter per column group, zero before the launch and zero again after it.
// The normed epilogues take the per-row RMSNorm scale from part_ss as the other GEMMs do.
constexpr int SPLITK_MAX = 8;
bool gemm_splitk_supported(int epi, int M, int ct);
hipError_t launch_gemm_splitk(int epi, int ct, int ksplit, const GemmArgs& a, float* part, unsigned* ctr,
                              hipStream_t s);
// Tiled GEMM for M > 64 (no second source): 128 x 128 output tiles.  Needs K % 32 == 0, an
// even k-step count and the A operand allocated for rows up to a multiple of
// gemm_tile_row_pad().  gemm_tile_parts gives the number of column groups (the argmax
// partials per row of the LM head).  ksplit > 1 (not for the LM head) cuts K into that many
// slices of whole stages (at most gemm_tile_stages): `part` holds gemm_tile_part_floats_per_wg()
// floats per (tile group, slice) and `ctr` one counter per tile group (gemm_tile_groups), zero
// before the launch and zero again after it.
bool gemm_tile_supported(int M, int K, int ksteps);
int gemm_tile_row_pad();
int gemm_tile_parts(int n_tiles);
int gemm_tile_groups(int M, int n_tiles);
int gemm_tile_stages(int ksteps);
size_t gemm_tile_part_floats_per_wg();
int gemm_tile_wgs_per_cu();   // workgroups of the tiled GEMM resident per CU
hipError_t launch_gemm_tile(int epi, const GemmArgs& a, int ksplit, float* part, unsigned* ctr, hipStream_t s);
// kh: key halves per stage (2 when the unit has at most 4 row tiles, else 1); 8 wavefronts per workgroup.
hipError_t launch_attention(int head_dim, int kh, int zslices, int units, const AttnArgs& a, hipStream_t s);
hipError_t launch_attention_combine(int head_dim, int units, int rows, const AttnArgs& a, hipStream_t s);
hipError_t launch_finish(const FinishArgs& a, hipStream_t s);
// Quadratic self-speculation: the ensemble verifier's per-chunk keys (0 < lambda < 1; grid
// batch*quad_k x ens_chunks), then acceptance, commit and the next speculative tokens (grid batch).
constexpr int ENS_CHUNKS = 32;
hipError_t launch_quad_ensemble(const FinishArgs& a, hipStream_t s);
hipError_t launch_quad_finish(const FinishArgs& a, hipStream_t s);

}  // namespace nld
