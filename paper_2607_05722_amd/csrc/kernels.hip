// HIP kernels of the block-decode step for gfx950 (CDNA4).
//
// One forward pass over a k-token block per sequence (arXiv 2607.05722,
// Sec. 3.3, linear self-speculation) is:
//   embed -> L x [QKV GEMM (RMSNorm fused into the operand load; RoPE and the
//                 K/V cache write fused into the epilogue),
//                 block-masked GQA attention over key splits (+ split merge),
//                 O GEMM (+ residual),
//                 gate/up GEMM (RMSNorm fused; SwiGLU epilogue),
//                 down GEMM (+ residual)]
//         -> LM-head GEMM (final RMSNorm fused; per-workgroup argmax keys)
//         -> per-sequence argmax + draft extraction / acceptance.
//
// The GEMMs are skinny (M = batch*k rows, usually 8..32): bound by streaming the
// bf16 weights from HBM.  Weights are pre-packed so that one 16-byte load per
// lane of a wavefront is exactly one MFMA B operand (1 KiB contiguous per
// wavefront load).
//
// Communication between workgroups of one launch.  The normed GEMM hands out
// tiles from a counter.  The split-K GEMM, the 17..64-row normed GEMM and the
// tiled GEMM with K slices meet through last-arriver counters; no workgroup ever
// waits for another.  The protocol of a slice partial:
//   1. every lane writes its part with agent-scope relaxed atomic stores;
//   2. s_waitcnt(0): the wavefront waits until each of its stores is
//      acknowledged, then a workgroup barrier;
//   3. one thread adds 1 to the counter (agent-scope relaxed fetch_add); the
//      workgroup that reads ksplit - 1 is the last to arrive;
//   4. the last arriver resets the counter to 0, reads the other partials with
//      agent-scope relaxed atomic loads, adds the slices in slice order (so the
//      sum does not depend on who arrived last) and runs the epilogue.
// Why this orders the data: agent-scope stores are made visible at agent scope
// (past the XCD-local L2) by the time they are acknowledged, so after step 2
// the partials are readable by agent-scope loads from any XCD; the barrier and
// the data dependence through the counter's value order step 4 after step 3.
// The C++ memory model would ask for an agent-scope release fence before the
// fetch_add (an L2 write-back measured at 11-18 us per kernel here); relaxed
// stores plus the store-acknowledgement wait rely instead on how gfx950
// completes agent-scope stores.  Repeated passes giving bit-identical results
// guard it in the tests.  Every counter is back at zero when its kernel ends,
// and the embedding kernel zeroes all of them at the start of each pass.

#include "nld_internal.h"

#include <hip/hip_ext.h>

#include <math.h>

namespace nld {

// Per-workgroup phase timestamps (a diagnostic build only, -DNLD_TIMELINE; see timeline.py): thread 0
// of each workgroup records the 100 MHz real-time counter at the phase boundaries of the kernels of
// one layer pass, class x workgroup x phase.  In the normal build NLD_TS expands to nothing.
#ifdef NLD_TIMELINE
__device__ unsigned long long g_timeline[8][8192][8];
#define NLD_TS(cls, ph)                                                                                   \
    do {                                                                                                  \
        if (threadIdx.x == 0)                                                                             \
            g_timeline[cls][blockIdx.x + blockIdx.y * gridDim.x + blockIdx.z * gridDim.x * gridDim.y][ph] = \
                __builtin_amdgcn_s_memrealtime();                                                         \
    } while (0)
#else
#define NLD_TS(cls, ph) do { } while (0)
#endif
enum TimelineClass { TL_QKV = 0, TL_ATTENTION = 1, TL_COMBINE = 2, TL_GATE_UP = 3, TL_O = 4, TL_DOWN = 5, TL_LM = 6 };

// Every kernel launch goes through here: a plain launch, or, while launch tracing is on,
// a launch whose start and stop events are recorded on the dispatch itself.
template <typename... KArgs, typename... Args>
static void launch(void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t s, Args... args) {
    hipEvent_t e0, e1;
    if (trace_launch_events(&e0, &e1)) hipExtLaunchKernelGGL(kernel, grid, block, 0, s, e0, e1, 0, args...);
    else kernel<<<grid, block, 0, s>>>(args...);
}


static constexpr uint32_t DEV_BAD_TOKEN = 0x1u;
static constexpr uint32_t DEV_CAPACITY = 0x2u;
static constexpr uint32_t DEV_BAD_LENGTH = 0x4u;
static constexpr uint32_t DEV_MASK_LEFT = 0x8u;

__device__ __forceinline__ int committed_length(const int32_t* lengths, int b, int max_len, uint32_t* status) {
    int p = lengths[b];
    if (p < 0) {
        atomicOr(status, DEV_BAD_LENGTH);
        p = 0;
    }
    return p < max_len ? p : max_len;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

__device__ __forceinline__ unsigned long long umax64(unsigned long long a, unsigned long long b) { return a > b ? a : b; }

// =====================================================================================
// GEMM epilogues, one output row per call.  A 16x16 output tile (packed column tile
// t) is finished by up to four wavefronts together: the wavefront that takes index i
// handles rows 4g + i of the tile (g = lane / 16) and lane 16g + r holds column r.
// y is the finished (RMSNorm-scaled) value of row m, column r.
// =====================================================================================
// pos: absolute position of row m (block row j at P_b + j).  RoPE uses the per-row
// (cos, sin) table built by the embedding kernel.
__device__ __forceinline__ void epi_qkv(const GemmArgs& a, float y, int m, int t, int lane, int pos) {
    const int r = lane & 15;
    const int D = a.head_dim;
    const int tiles_per_head = D / 16;
    const int hh = t / tiles_per_head, u = t % tiles_per_head;
    const int fi = 8 * u + (r & 7);             // rotary frequency index, < D/2
    const int dim = (r < 8) ? fi : D / 2 + fi;  // lanes r and r^8 hold the pair (fi, fi + D/2)
    const int nq = a.n_q_heads, nkv = a.n_kv_heads;
    const int kind = hh < nq ? 0 : (hh < nq + nkv ? 1 : 2);
    const bool ok = m < a.M;
    const float partner = __shfl_xor(y, 8);
    float out = y;
    if (kind < 2) {
        const float2 cs = a.rope[(size_t)(ok ? m : 0) * (D / 2) + fi];
        out = (r < 8) ? (y * cs.x - partner * cs.y) : (y * cs.x + partner * cs.y);
    }
    if (!ok) return;
    const int b = m / a.k_blk, jb = m - b * a.k_blk;
    if (kind == 0) {
        const int G = nq / nkv;
        const int row = (hh % G) * a.k_blk + jb;
        store_split(a.q_out, q_index(b * nkv + hh / G, row, dim, a.q_row_tiles, D), out, a.plain & SITE_Q);
        return;
    }
    // K/V: split into the block buffer (what this pass's attention over the block's
    // own keys reads) and, in a verify pass, bf16 into the cache (what a commit keeps)
    const int kvh = hh - nq - (kind == 2 ? nkv : 0);
    const size_t unit = (size_t)b * nkv + kvh;
    const uint16_t ob = (uint16_t)f32_to_bf16(out);
    const uint16_t lo = (a.plain & SITE_KV) ? (uint16_t)0 : (uint16_t)f32_to_bf16(out - bf16_to_f32(ob));
    if (kind == 1) {
        a.blk_k[(unit * 2 * 64 + jb) * D + dim] = ob;
        a.blk_k[((unit * 2 + 1) * 64 + jb) * D + dim] = lo;
    } else {
        a.blk_v[(unit * 2 * D + dim) * 64 + jb] = ob;
        a.blk_v[((unit * 2 + 1) * D + dim) * 64 + jb] = lo;
    }
    if (!a.write_cache) return;
    if (a.quad_k > 0 && jb >= a.quad_k) return;   // quadratic layout: only the chain rows are AR rows
    if (pos >= a.max_len) atomicOr(a.status, DEV_CAPACITY);
    else if (kind == 1) a.kc[(unit * a.max_len + pos) * D + dim] = ob;
    else a.vc[((unit * (a.max_len / 64) + pos / 64) * D + dim) * 64 + (pos & 63)] = ob;
}

__device__ __forceinline__ void epi_swiglu(const GemmArgs& a, float y, int m, int t, int lane) {
    const int r = lane & 15;
    const int col = 8 * t + (r & 7);
    const float partner = __shfl_xor(y, 8);   // lanes r < 8 hold gate columns, r^8 the matching up columns
    if (m < a.M && r < 8 && col < a.ffn) {
        const float act = y / (1.0f + expf(-y)) * partner;
        store_split(a.act, split_index(m, col, (a.ffn + 31) / 32), act, a.plain & SITE_ACT);
    }
}

// Softmax statistics as (max, sum of exp(z - max)); (-inf, 0) is the empty set.
__device__ __forceinline__ float2 lse_merge(float2 a, float2 b) {
    if (b.x == -INFINITY) return a;
    if (a.x == -INFINITY) return b;
    const float mx = fmaxf(a.x, b.x);
    return float2{mx, a.y * expf(a.x - mx) + b.y * expf(b.x - mx)};
}

// Returns, in every lane, the argmax key of row m over this tile's 16 columns and,
// when the pass asks for softmax statistics, the tile row's (max, sum of exp) in
// *lse.  The excluded column (the mask token when denoising) takes part in neither.
__device__ __forceinline__ unsigned long long epi_lmhead(const GemmArgs& a, float y, int m, int t, int lane,
                                                         float2* lse) {
    const int r = lane & 15;
    const int n = t * 16 + r;
    const bool in = m < a.M && n < a.vocab;
    const bool ok = in && n != a.exclude_id;
    if (in && a.logits) a.logits[(size_t)m * a.vocab + n] = y;
    if (in && a.ens_logits) {   // quadratic layout: the verifier rows (chain row i, mask 1 of group i)
        const int b = m / a.k_blk, jb = m - b * a.k_blk, qk = a.quad_k;
        const int ci = jb < qk ? jb : ((jb - qk) % qk == 0 ? qk + (jb - qk) / qk : -1);
        if (ci >= 0) a.ens_logits[((size_t)b * 2 * qk + ci) * a.vocab + n] = y;
    }
    unsigned long long key = ok ? argmax_key(y, (uint32_t)n) : 0ull;
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) key = umax64(key, __shfl_xor(key, off));
    if (a.part_lse) {
        float mx = ok ? y : -INFINITY;
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        float e = ok ? expf(y - mx) : 0.f;
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) e += __shfl_xor(e, off);
        *lse = float2{mx, e};
    }
    return key;
}

// xres: the residual x[m][16t + r]; gn: the next RMSNorm's gain at column 16t + r.
// Writes x += v, the next RMSNorm's split operand x * gain_next and the row's sum of
// x^2 over the tile's 16 columns.
__device__ __forceinline__ void epi_resid(const GemmArgs& a, float v, int m, int t, int lane, float xres, float gn) {
    const int r = lane & 15;
    const int N = a.n_tiles * 16;
    const int n = t * 16 + r;
    const bool ok = m < a.M;
    const float xn = xres + v;
    if (ok) {
        a.x[(size_t)m * N + n] = xn;
        store_split(a.xg_out, split_index(m, n, N / 32), xn * gn, a.plain & (SITE_NORM | SITE_FINAL));
    }
    float sq = ok ? xn * xn : 0.f;
    sq += __shfl_xor(sq, 1);
    sq += __shfl_xor(sq, 2);
    sq += __shfl_xor(sq, 4);
    sq += __shfl_xor(sq, 8);
    if (r == 0 && ok) a.part_ss_out[(size_t)m * a.n_tiles + t] = sq;
}

// 1/rms for `rows` rows starting at m0 from the producer's 16-column partial sums
// (fixed summation order); rows past M get 0.  One wavefront per row.
__device__ __forceinline__ void rms_scales(const GemmArgs& a, int m0, int rows, float* inv_s) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    for (int rr = wave; rr < rows; rr += nw) {
        const int m = m0 + rr;
        float s = 0.f;
        if (m < a.M) {
            const float* ps = a.part_ss + (size_t)m * a.n_ss;
            for (int p = lane; p < a.n_ss; p += 64) s += ps[p];
        }
        s = wave_sum(s);
        if (lane == 0) inv_s[rr] = (m < a.M) ? 1.0f / sqrtf(s / (float)a.K + a.eps) : 0.f;
    }
}

// =====================================================================================
// Normed multi-tile GEMM (M <= 16 rows).  A workgroup of NW wavefronts owns a
// contiguous range of output tiles; wavefront w owns the reduction slice
// [32*KS*w, 32*KS*(w+1)).  At the start each wavefront loads its slice of the
// split operand bf16(x * gain) (hi and lo) and keeps it in registers for all
// tiles; the per-row RMSNorm scale comes from the producer's partial sums of
// squares.  Weights stream through one register buffer: the load of the next
// tile's step s is issued as soon as step s of the current tile has been
// multiplied, so one tile's worth of loads is in flight throughout.  Per tile
// the NW partial products meet in LDS and one wavefront (rotating) runs the
// epilogue.
// =====================================================================================
template <int KS, int EPI>
__global__ void __launch_bounds__(KS >= 16 ? 512 : 1024) gemm_norm_kernel(GemmArgs a) {
    __shared__ f32x4_t red[2][16][64];
    __shared__ float inv_s[16];
    __shared__ unsigned long long key_s[16][16];
    __shared__ float2 lse_s[16][16];
    __shared__ int pos_s[16];

    __shared__ int next_s[2];

    constexpr int TLC = EPI == EPI_QKV ? TL_QKV : (EPI == EPI_SWIGLU ? TL_GATE_UP : TL_LM);
    NLD_TS(TLC, 0);
    const int NW = blockDim.x >> 6;
    if constexpr (EPI == EPI_LMHEAD) {
        if (threadIdx.x < 256) {
            key_s[threadIdx.x >> 4][threadIdx.x & 15] = 0ull;
            lse_s[threadIdx.x >> 4][threadIdx.x & 15] = float2{-INFINITY, 0.f};
        }
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int T = a.n_tiles, G = gridDim.x;
    const int s0 = wave * KS;

    // Tiles are handed out dynamically: workgroup b starts with tile b, further tiles
    // come from a counter (tile index G + counter), requested one tile ahead so that
    // the atomic's latency hides behind the current tile.  Faster workgroups (and
    // XCDs) end up with more tiles.
    int cur = blockIdx.x;
    unsigned grab = 0u;
    if (threadIdx.x == 0 && G < T) grab = atomicAdd(a.tile_ctr, 1u);

    // operand slice: row r, columns 32*(s0+s) + 8g .. +8, hi and lo.  Requested before the first
    // weight tile: loads complete in issue order, and the operand (L2 hits after the first workgroups)
    // then no longer waits behind the tile's HBM reads (8B shapes, k = 16: QKV 16.7 against 17.5 us,
    // gate/up 37.8 against 39.4 us, LM head 198.5 against 200.5 us).
    uint4 ah[KS], al[KS];
    const bool row_ok = r < a.M;
    const uint16_t* ar = a.A + (size_t)s0 * 1024 + (size_t)lane * 8;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        ah[s] = row_ok ? *(const uint4*)(ar + (size_t)s * 1024) : uint4{0u, 0u, 0u, 0u};
        al[s] = row_ok ? *(const uint4*)(ar + (size_t)s * 1024 + SPLIT_LO) : uint4{0u, 0u, 0u, 0u};
    }
    uint4 wb[KS];
    if (cur < T) {
        const uint4* p = a.W + ((size_t)cur * a.ksteps + s0) * 64 + lane;
#pragma unroll
        for (int s = 0; s < KS; ++s) wb[s] = load_stream(p + (size_t)s * 64);
    }
    rms_scales(a, 0, 16, inv_s);
    if constexpr (EPI == EPI_QKV) {
        if (threadIdx.x < 16) {   // absolute position of block row m: P_b + j
            const int m = min((int)threadIdx.x, a.M - 1);
            pos_s[threadIdx.x] = committed_length(a.lengths, m / a.k_blk, a.max_len, a.status) + m % a.k_blk;
        }
    }
    if (threadIdx.x == 0) next_s[0] = G < T ? min(G + (int)grab, T) : T;
    __syncthreads();

    // A tile is finished by FIN wavefronts (wavefront i of the group takes rows 4g + i,
    // 4g + i + FIN, ...); the groups take the tiles in turn.
    NLD_TS(TLC, 1);   // operand, first tile and row statistics in
    const int FIN = NW < 4 ? NW : 4, groups = NW / FIN;
    for (int it = 0; cur < T; ++it) {
        const int t = cur;
        const int nxt = next_s[it & 1];   // its weights stream in while tile t is multiplied
        if (threadIdx.x == 0 && nxt < T) grab = atomicAdd(a.tile_ctr, 1u);
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f}, accl = {0.f, 0.f, 0.f, 0.f};
        const bool more = nxt < T;
        const uint4* p = a.W + ((size_t)nxt * a.ksteps + s0) * 64 + lane;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            acc = mfma_16x16x32(ah[s], wb[s], acc);
            accl = mfma_16x16x32(al[s], wb[s], accl);
            if (more) wb[s] = load_stream(p + (size_t)s * 64);
        }
        if (threadIdx.x == 0) next_s[(it + 1) & 1] = nxt < T ? min(G + (int)grab, T) : T;
        const int parity = it & 1;
        red[parity][wave][lane] = acc + accl;
        __syncthreads();
        cur = nxt;
        if (wave / FIN == it % groups) {
            const float* rp = (const float*)&red[parity][0][lane];
            for (int i = wave % FIN; i < 4; i += FIN) {
                float v = rp[i];
                for (int w = 1; w < NW; ++w) v += rp[w * 256 + i];   // fixed order over the K-slices
                const int m = 4 * g + i;
                const float y = v * inv_s[m];
                if constexpr (EPI == EPI_QKV) epi_qkv(a, y, m, t, lane, pos_s[m]);
                else if constexpr (EPI == EPI_SWIGLU) epi_swiglu(a, y, m, t, lane);
                else {
                    float2 tl;
                    const unsigned long long key = epi_lmhead(a, y, m, t, lane, &tl);
                    if (r == 0) {
                        key_s[wave][m] = umax64(key_s[wave][m], key);
                        if (a.part_lse) lse_s[wave][m] = lse_merge(lse_s[wave][m], tl);
                    }
                }
            }
        }
    }

    NLD_TS(TLC, 2);
    if constexpr (EPI == EPI_LMHEAD) {
        // one argmax key per row for this workgroup
        __syncthreads();
        if ((int)threadIdx.x < a.M && threadIdx.x < 16) {
            unsigned long long best = 0ull;
            for (int w = 0; w < NW; ++w) best = umax64(best, key_s[w][threadIdx.x]);
            a.part_keys[(size_t)threadIdx.x * a.n_parts + blockIdx.x] = best;
            if (a.part_lse) {
                float2 st = float2{-INFINITY, 0.f};
                for (int w = 0; w < NW; ++w) st = lse_merge(st, lse_s[w][threadIdx.x]);
                a.part_lse[(size_t)threadIdx.x * a.n_parts + blockIdx.x] = st;
            }
        }
    }
}

bool gemm_norm_supported(int ks) { return ks == 4 || ks == 8 || ks == 16 || ks == 20; }

template <int KS>
static hipError_t launch_norm_ks(int epi, int waves, int grid, const GemmArgs& a, hipStream_t s) {
    const dim3 blk(waves * 64);
    switch (epi) {
        case EPI_QKV: launch(gemm_norm_kernel<KS, EPI_QKV>, dim3(grid), dim3(blk), s, a); break;
        case EPI_SWIGLU: launch(gemm_norm_kernel<KS, EPI_SWIGLU>, dim3(grid), dim3(blk), s, a); break;
        case EPI_LMHEAD: launch(gemm_norm_kernel<KS, EPI_LMHEAD>, dim3(grid), dim3(blk), s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

int gemm_norm_max_waves(int ks) { return ks >= 16 ? 8 : 16; }

hipError_t launch_gemm_norm(int epi, int ks, int waves, int grid, const GemmArgs& a, hipStream_t s) {
    if (waves < 1 || waves > gemm_norm_max_waves(ks)) return hipErrorInvalidValue;
    switch (ks) {
        case 4: return launch_norm_ks<4>(epi, waves, grid, a, s);
        case 8: return launch_norm_ks<8>(epi, waves, grid, a, s);
        case 16: return launch_norm_ks<16>(epi, waves, grid, a, s);
        case 20: return launch_norm_ks<20>(epi, waves, grid, a, s);
        default: return hipErrorInvalidValue;
    }
}

// =====================================================================================
// Normed multi-tile GEMM for 17..64 rows (QKV, gate/up, LM head of a pass with two or four
// row tiles, such as the quadratic self-speculation pass).  The operand of MT row tiles is
// too large to reload per column tile (the split operand is 2 KB per row tile and k-step,
// against 1 KB of weights per column tile), so a workgroup of 8 wavefronts holds one K
// slice of it in registers for every column tile it multiplies: wavefront w owns k-steps
// [(ks*8 + w)*KS, +KS) of slice ks = blockIdx.y.  Workgroup x of a slice takes column tiles
// x, x + gridDim.x, ...; their weights stream through PF register buffers, each refilled
// with the tile PF ahead as soon as it has been multiplied.  Per tile the wavefronts'
// products meet in LDS and the slice's partial goes to the workspace with agent-scope
// stores.  After its last tile the workgroup counts itself in on each tile's counter; the
// workgroup that completes a tile reads the slices' partials in slice order and runs the
// epilogue (wavefront w takes row tile w % MT of every (8/MT)-th completed tile), then
// resets the counter.
// =====================================================================================
constexpr int NK_MAXT = 160;   // column tiles per workgroup (the host keeps ceil(n_tiles / grid.x) within it)

template <int MT, int KS, int PF, int EPI>
__global__ void __launch_bounds__(512) gemm_normk_kernel(GemmArgs a, float* part, unsigned* tctr, int ksplit) {
    constexpr int NW = 8;
    constexpr int WPR = NW / MT;   // wavefronts per row tile in the epilogue
    static_assert(NW % MT == 0, "row tiles must divide the wavefronts");
    __shared__ f32x4_t red[2][NW][MT][64];
    __shared__ float inv_s[16 * MT];
    __shared__ unsigned char last_s[NK_MAXT];
    __shared__ int fin_s[NK_MAXT];
    __shared__ int nfin_s;
    __shared__ unsigned long long key_s[NW][16];
    __shared__ float2 lse_s[NW][16];
    typedef unsigned long long u64;
    constexpr int TLC = EPI == EPI_QKV ? TL_QKV : (EPI == EPI_SWIGLU ? TL_GATE_UP : TL_LM);
    NLD_TS(TLC, 0);

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int x = blockIdx.x, Gx = gridDim.x, ks = blockIdx.y;
    const int T = a.n_tiles;
    const int nt = x < T ? (T - 1 - x) / Gx + 1 : 0;
    const int s0 = (ks * NW + wave) * KS;
    const uint4 zero4 = {0u, 0u, 0u, 0u};

    // this wavefront's operand slice, hi and lo, for every row tile
    uint4 ah[MT][KS], al[MT][KS];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            const int ss = s0 + s;
            const bool ok = mt * 16 + r < a.M && ss < a.ksteps && ss * 32 + 8 * g < a.K;
            const uint16_t* ap = a.A + (size_t)(mt * a.ksteps + ss) * 1024 + (size_t)lane * 8;
            ah[mt][s] = zero4;
            al[mt][s] = zero4;
            if (ok) {
                ah[mt][s] = *(const uint4*)ap;
                al[mt][s] = *(const uint4*)(ap + SPLIT_LO);
            }
        }

    rms_scales(a, 0, 16 * MT, inv_s);   // visible after the first barrier below
    if constexpr (EPI == EPI_LMHEAD) {
        if (threadIdx.x < NW * 16) {
            key_s[threadIdx.x / 16][threadIdx.x % 16] = 0ull;
            lse_s[threadIdx.x / 16][threadIdx.x % 16] = float2{-INFINITY, 0.f};
        }
    }
    if (nt == 0) return;   // no column tile here (the whole workgroup leaves; the LM head writes no key)

    // Per tile, every wavefront stores EL elements of one row tile's partial: row tile w % MT,
    // elements (w / MT) * EL .. +EL of each lane's four (one 8-byte store, or one 4-byte store).
    constexpr int EL = 4 / WPR;
    static_assert(EL == 1 || EL == 2, "one 4- or 8-byte partial store per wavefront and tile");
    const int st_mt = wave % MT, st_e0 = (wave / MT) * EL;
    auto store_part = [&](int t, f32x4_t v) __attribute__((always_inline)) {
        float* pp = part + ((((size_t)t * ksplit + ks) * MT + st_mt) * 64 + lane) * 4 + st_e0;
        if constexpr (EL == 2)
            __hip_atomic_store((u64*)pp, __builtin_bit_cast(u64, f32x2_t{v[st_e0], v[st_e0 + 1]}), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        else
            __hip_atomic_store(pp, v[st_e0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };

    // Weight loads are unconditional, with the tile and the k-step clamped into the matrix (a
    // k-step past the end meets a zero operand; a tile past the workgroup's last is never
    // multiplied).  Each buffer's loads are followed by one partial store, here a zero into the
    // first tile's slot that its real partial overwrites later, so that the prologue leaves the
    // same sequence of outstanding loads and stores as a loop iteration: the wait counts then
    // stay exact and the next PF tiles' loads remain in flight across the loop.
    const int s_last = a.ksteps - 1;
    uint4 wb[PF][KS];
#pragma unroll
    for (int p = 0; p < PF; ++p) {
#pragma unroll
        for (int s = 0; s < KS; ++s)
            wb[p][s] = load_stream(a.W + ((size_t)min(x + p * Gx, T - 1) * a.ksteps + min(s0 + s, s_last)) * 64 + lane);
        store_part(x, f32x4_t{0.f, 0.f, 0.f, 0.f});
    }

    // epilogue of row tile mt of tile t from its full sum v (lane layout of an MFMA result);
    // LM head: the row maxima and statistics accumulate per wavefront in LDS (rows 4g + i)
    auto epilogue = [&](f32x4_t v, int t, int mt) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int m = 16 * mt + 4 * g + i;
            const float y = v[i] * inv_s[m];
            if constexpr (EPI == EPI_QKV) {
                const int mc = min(m, a.M - 1);
                const int pos = committed_length(a.lengths, mc / a.k_blk, a.max_len, a.status) + mc % a.k_blk;
                epi_qkv(a, y, m, t, lane, pos);
            } else if constexpr (EPI == EPI_SWIGLU) {
                epi_swiglu(a, y, m, t, lane);
            } else {
                float2 tl;
                const u64 key = epi_lmhead(a, y, m, t, lane, &tl);
                if (r == 0) {
                    key_s[wave][4 * g + i] = umax64(key_s[wave][4 * g + i], key);
                    if (a.part_lse) lse_s[wave][4 * g + i] = lse_merge(lse_s[wave][4 * g + i], tl);
                }
            }
        }
    };

    // tile j (the workgroup's j-th) from buffer p, whose next tile is j + PF
    auto tile = [&](int j, int p_dummy, uint4 (&w)[KS]) __attribute__((always_inline)) {
        (void)p_dummy;
        const int t = x + j * Gx;
        f32x4_t acc[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        const int tn = min(x + (j + PF) * Gx, T - 1);
#pragma unroll
        for (int s = 0; s < KS; ++s) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                acc[mt] = mfma_16x16x32(ah[mt][s], w[s], acc[mt]);
                acc[mt] = mfma_16x16x32(al[mt][s], w[s], acc[mt]);
            }
            w[s] = load_stream(a.W + ((size_t)tn * a.ksteps + min(s0 + s, s_last)) * 64 + lane);
        }
        const int par = j & 1;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) red[par][wave][mt][lane] = acc[mt];
        __syncthreads();
        // the slice's partial: this wavefront's elements of row tile st_mt (fixed order over
        // the wavefronts)
        f32x4_t v = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int w2 = 0; w2 < NW; ++w2) v += red[par][w2][st_mt][lane];
        store_part(t, v);
    };
    // whole groups of PF tiles with no condition inside, so the loop keeps one shape; then the rest
    int j0 = 0;
    for (; j0 + PF <= nt; j0 += PF) {
#pragma unroll
        for (int p = 0; p < PF; ++p) tile(j0 + p, p, wb[p]);
    }
#pragma unroll
    for (int p = 0; p < PF - 1; ++p)
        if (j0 + p < nt) tile(j0 + p, p, wb[p]);

    NLD_TS(TLC, 1);   // main loop done
    {   // the tiles this workgroup completes (with a single slice: all of its own)
        // every lane's partial stores are acknowledged before the workgroup counts itself in
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_s_waitcnt(0);
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __syncthreads();
        for (int j = threadIdx.x; j < nt; j += blockDim.x)
            last_s[j] = __hip_atomic_fetch_add(tctr + x + j * Gx, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                        (unsigned)(ksplit - 1);
        __syncthreads();
        if (threadIdx.x == 0) {
            int n = 0;
            for (int j = 0; j < nt; ++j)
                if (last_s[j]) fin_s[n++] = x + j * Gx;
            nfin_s = n;
        }
        __syncthreads();
        const int nfin = nfin_s;
        for (int c = threadIdx.x; c < nfin; c += blockDim.x)
            __hip_atomic_exchange(tctr + fin_s[c], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        // wavefront w: row tile w % MT of completed tiles w / MT, + WPR, ...; two tiles' partials in flight
        const int mt = wave % MT;
        for (int c = wave / MT; c < nfin; c += 2 * WPR) {
            const int c2 = c + WPR;
            const int ta = fin_s[c], tb = c2 < nfin ? fin_s[c2] : ta;
            f32x4_t va = {0.f, 0.f, 0.f, 0.f}, vb = {0.f, 0.f, 0.f, 0.f};
            for (int sl = 0; sl < ksplit; ++sl) {
                const u64* qa = (const u64*)(part + ((((size_t)ta * ksplit + sl) * MT + mt) * 64 + lane) * 4);
                const u64* qb = (const u64*)(part + ((((size_t)tb * ksplit + sl) * MT + mt) * 64 + lane) * 4);
                const f32x2_t a0 = __builtin_bit_cast(f32x2_t, __hip_atomic_load(qa, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
                const f32x2_t a1 = __builtin_bit_cast(f32x2_t, __hip_atomic_load(qa + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
                const f32x2_t b0 = __builtin_bit_cast(f32x2_t, __hip_atomic_load(qb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
                const f32x2_t b1 = __builtin_bit_cast(f32x2_t, __hip_atomic_load(qb + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
                va += f32x4_t{a0[0], a0[1], a1[0], a1[1]};
                vb += f32x4_t{b0[0], b0[1], b1[0], b1[1]};
            }
            epilogue(va, ta, mt);
            if (c2 < nfin) epilogue(vb, tb, mt);
        }
    }
    NLD_TS(TLC, 2);   // completed tiles finished

    if constexpr (EPI == EPI_LMHEAD) {
        // one argmax key (and softmax statistics) per row for this workgroup
        __syncthreads();
        if ((int)threadIdx.x < 16 * MT) {
            const int m = threadIdx.x, mt = m / 16, rl = m % 16;
            if (m < a.M) {
                u64 k2 = 0ull;
                float2 st = float2{-INFINITY, 0.f};
                for (int w = mt; w < NW; w += MT) {   // the wavefronts that finished row tile mt
                    k2 = umax64(k2, key_s[w][rl]);
                    st = lse_merge(st, lse_s[w][rl]);
                }
                const int part_id = x + Gx * ks;
                a.part_keys[(size_t)m * a.n_parts + part_id] = k2;
                if (a.part_lse) a.part_lse[(size_t)m * a.n_parts + part_id] = st;
            }
        }
    }
}

bool gemm_normk_supported(int epi, int M) {
    return (epi == EPI_QKV || epi == EPI_SWIGLU || epi == EPI_LMHEAD) && M > 16 && M <= 64;
}

// k-steps per slice: 8 wavefronts x 4 (four row tiles) or x 8 (two row tiles)
int gemm_normk_kstep_span(int M) { return 8 * (M > 32 ? 4 : 8); }

int gemm_normk_max_tiles() { return NK_MAXT; }

template <int MT, int KS>
static hipError_t launch_normk_mt(int epi, dim3 grid, const GemmArgs& a, float* part, unsigned* tctr, int ksplit,
                                  hipStream_t s) {
    constexpr int PF = MT >= 4 ? 3 : 2;   // tiles of weights in flight per wavefront (registers permitting)
    switch (epi) {
        case EPI_QKV: launch(gemm_normk_kernel<MT, KS, PF, EPI_QKV>, grid, dim3(512), s, a, part, tctr, ksplit); break;
        case EPI_SWIGLU: launch(gemm_normk_kernel<MT, KS, PF, EPI_SWIGLU>, grid, dim3(512), s, a, part, tctr, ksplit); break;
        case EPI_LMHEAD: launch(gemm_normk_kernel<MT, KS, PF, EPI_LMHEAD>, grid, dim3(512), s, a, part, tctr, ksplit); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_gemm_normk(int epi, int grid_x, const GemmArgs& a, float* part, unsigned* tctr, hipStream_t s) {
    if (!gemm_normk_supported(epi, a.M) || grid_x < 1) return hipErrorInvalidValue;
    if ((a.n_tiles + grid_x - 1) / grid_x > NK_MAXT) return hipErrorInvalidValue;
    const int span = gemm_normk_kstep_span(a.M);
    const int ksplit = (a.ksteps + span - 1) / span;
    const dim3 grid((unsigned)grid_x, (unsigned)ksplit);
    if (a.M > 32) return launch_normk_mt<4, 4>(epi, grid, a, part, tctr, ksplit, s);
    return launch_normk_mt<2, 8>(epi, grid, a, part, tctr, ksplit, s);
}

// =====================================================================================
// Streamed GEMM: out[m][n] = sum_k A[m][k] W[n][k] for 16*MT rows x 16*CT columns per
// workgroup; the NW wavefronts split the reduction, each streaming its slice of the
// weights and of the bf16 activations with one batch in flight ahead of the MFMAs.
// Every operand is split (two MFMAs per weight operand).  Used for the O and down
// projections (residual epilogue) and, for M > 16, for every projection (the
// per-row RMSNorm scale is then formed in the prologue).
// =====================================================================================
template <int MT, int CT, bool SPLIT, int NW = 8>
struct Batch {
    static constexpr int OPS = CT + MT * (SPLIT ? 2 : 1);   // operand quads per k-step
    // 16 wavefronts (1024 threads, at most 128 registers each): half the batch
    static constexpr int U = ((OPS <= 3) ? 8 : ((OPS <= 5) ? 4 : 2)) / (NW > 8 ? 2 : 1);
    uint4 w[U][CT];
    uint4 x[U][MT];
    uint4 xl[SPLIT ? U : 1][SPLIT ? MT : 1];
};

template <int MT, int CT, int NW, int EPI, bool XK>
__global__ void __launch_bounds__(NW * 64) gemm_stream_kernel(GemmArgs a) {
    constexpr bool SPLIT = true;
    constexpr bool NORMED = EPI == EPI_QKV || EPI == EPI_SWIGLU || EPI == EPI_LMHEAD;
    typedef Batch<MT, CT, SPLIT, NW> B;
    constexpr int U = B::U;
    constexpr int BSTRIDE = SPLIT ? 1024 : 512;   // elements per (row tile, k-step) block
    __shared__ f32x4_t red[NW][MT * CT][64];
    __shared__ unsigned long long key_s[16 * MT];
    __shared__ float2 lse_s[16 * MT][CT];
    __shared__ float inv_s[16 * MT];
    NLD_TS(TL_O, 0);

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int t0 = blockIdx.x * CT;
    const int m0 = blockIdx.y * 16 * MT;

    const int per = (a.ksteps + NW - 1) / NW;
    const int s_begin = min(a.ksteps, wave * per);
    const int s_end = min(a.ksteps, s_begin + per);

    const uint4* wp[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
        const int t = min(t0 + ct, a.n_tiles - 1);
        wp[ct] = a.W + (size_t)t * a.ksteps * 64 + lane;
    }
    const uint16_t* ap[MT];
    bool aok[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        aok[mt] = m0 + mt * 16 + r < a.M;
        ap[mt] = a.A + (size_t)(blockIdx.y * MT + mt) * a.ksteps * BSTRIDE + (size_t)lane * 8;
    }
    // XK: the second source's k-steps (W2 against A2) go one to a wavefront (wavefront w takes step
    // w, then w + NW, ...).  They are loaded before the main stream and multiplied after it, so the
    // main loop is the same as without them.
    constexpr int XS = XK ? 2 : 1;   // second-source k-steps held per wavefront (at most 2 * NW in all)
    uint4 xw[XS][CT], xa[XS][MT], xal[XS][MT];
    if constexpr (XK) {
#pragma unroll
        for (int i = 0; i < XS; ++i) {
            const int s2 = wave + i * NW;
            const bool in = s2 < a.ksteps2;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                const int t = min(t0 + ct, a.n_tiles - 1);
                xw[i][ct] = in ? a.W2[((size_t)t * a.ksteps2 + s2) * 64 + lane] : uint4{0u, 0u, 0u, 0u};
            }
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const uint16_t* ap2 = a.A2 + ((size_t)(blockIdx.y * MT + mt) * a.ksteps2 + s2) * BSTRIDE + (size_t)lane * 8;
                const bool ok = in && aok[mt];
                xa[i][mt] = ok ? *(const uint4*)ap2 : uint4{0u, 0u, 0u, 0u};
                xal[i][mt] = ok ? *(const uint4*)(ap2 + SPLIT_LO) : uint4{0u, 0u, 0u, 0u};
            }
        }
    }

    f32x4_t acc[MT][CT], accl[SPLIT ? MT : 1][SPLIT ? CT : 1];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[mt][ct] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if constexpr (SPLIT) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) accl[mt][ct] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }

    // Epilogue assignment: a tile is finished by FIN = 4 wavefronts, wavefront i of the
    // group taking rows 4g + i; the NW / 4 groups take the MT x CT tiles in turn.
    constexpr int FIN = 4, GROUPS = NW / FIN;
    static_assert(NW % FIN == 0, "wavefront count must be a multiple of 4");
    const int fi_row = wave % FIN, ti0 = wave / FIN;
    // residual value and next gain for this wavefront's first epilogue row, fetched up
    // front so that the epilogue waits on no load
    float xres0 = 0.f, gn0 = 0.f;
    if constexpr (EPI == EPI_RESID) {
        if (ti0 < MT * CT) {
            const int mt = ti0 / CT, ct = ti0 % CT;
            const int m = m0 + 16 * mt + 4 * g + fi_row;
            if (t0 + ct < a.n_tiles) {
                gn0 = bf16_to_f32(a.gain_next[(t0 + ct) * 16 + r]);
                if (m < a.M) xres0 = a.x[(size_t)m * a.n_tiles * 16 + (t0 + ct) * 16 + r];
            }
        }
    }

    const uint4 zero4 = {0u, 0u, 0u, 0u};
    auto load = [&](int s, B& buf) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int ss = s + u;
            const bool in = ss < s_end;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) buf.w[u][ct] = in ? wp[ct][(size_t)ss * 64] : zero4;
            const int kcol = ss * 32 + 8 * g;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const bool ok = in && aok[mt] && kcol < a.K;
                buf.x[u][mt] = ok ? *(const uint4*)(ap[mt] + (size_t)ss * BSTRIDE) : zero4;
                if constexpr (SPLIT) buf.xl[u][mt] = ok ? *(const uint4*)(ap[mt] + (size_t)ss * BSTRIDE + SPLIT_LO) : zero4;
            }
        }
    };
    auto compute = [&](const B& buf) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int ct = 0; ct < CT; ++ct) {
                    acc[mt][ct] = mfma_16x16x32(buf.x[u][mt], buf.w[u][ct], acc[mt][ct]);
                    if constexpr (SPLIT) accl[mt][ct] = mfma_16x16x32(buf.xl[u][mt], buf.w[u][ct], accl[mt][ct]);
                }
    };

    B b0, b1;
    load(s_begin, b0);
    if constexpr (NORMED) rms_scales(a, m0, 16 * MT, inv_s);   // visible after the barrier below
    for (int s = s_begin; s < s_end; s += 2 * U) {
        load(s + U, b1);
        compute(b0);
        load(s + 2 * U, b0);
        compute(b1);
    }

    NLD_TS(TL_O, 1);   // main loop done
    if constexpr (XK) {
#pragma unroll
        for (int i = 0; i < XS; ++i)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int ct = 0; ct < CT; ++ct) {
                    acc[mt][ct] = mfma_16x16x32(xa[i][mt], xw[i][ct], acc[mt][ct]);
                    accl[mt][ct] = mfma_16x16x32(xal[i][mt], xw[i][ct], accl[mt][ct]);
                }
    }
    if constexpr (SPLIT) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) acc[mt][ct] += accl[mt][ct];
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) red[wave][mt * CT + ct][lane] = acc[mt][ct];
    if constexpr (EPI == EPI_LMHEAD) {
        if (threadIdx.x < 16 * MT) key_s[threadIdx.x] = 0ull;
        if (threadIdx.x < 16 * MT * CT) lse_s[threadIdx.x / CT][threadIdx.x % CT] = float2{-INFINITY, 0.f};
    }
    __syncthreads();
    for (int ti = ti0; ti < MT * CT; ti += GROUPS) {
        const float* rp = (const float*)&red[0][ti][lane];
        float v = rp[fi_row];
#pragma unroll
        for (int w = 1; w < NW; ++w) v += rp[w * MT * CT * 256 + fi_row];   // fixed order over the K-slices
        const int mt = ti / CT, ct = ti % CT;
        const int t = t0 + ct;
        if (t >= a.n_tiles) continue;
        const int ml = 16 * mt + 4 * g + fi_row;   // row within the workgroup's rows
        const int m = m0 + ml;
        if constexpr (EPI == EPI_RESID) {
            float xr = xres0, gn = gn0;
            if (ti != ti0) {
                xr = m < a.M ? a.x[(size_t)m * a.n_tiles * 16 + t * 16 + r] : 0.f;
                gn = bf16_to_f32(a.gain_next[t * 16 + r]);
            }
            epi_resid(a, v, m, t, lane, xr, gn);
        } else if constexpr (EPI == EPI_QKV) {
            const int mc = min(m, a.M - 1);
            const int pos = committed_length(a.lengths, mc / a.k_blk, a.max_len, a.status) + mc % a.k_blk;
            epi_qkv(a, v * inv_s[ml], m, t, lane, pos);
        } else if constexpr (EPI == EPI_SWIGLU) {
            epi_swiglu(a, v * inv_s[ml], m, t, lane);
        } else if constexpr (EPI == EPI_SPLIT) {
            if (m < a.M) store_split(a.xg_out, split_index(m, t * 16 + r, a.n_tiles / 2), a.out_scale * v);
        } else {
            float2 tl;
            const unsigned long long key = epi_lmhead(a, v * inv_s[ml], m, t, lane, &tl);
            if (r == 0) {
                atomicMax(&key_s[ml], key);
                if (a.part_lse) lse_s[ml][ct] = tl;   // each (row, column tile) is finished once
            }
        }
    }
    if constexpr (EPI == EPI_LMHEAD) {
        __syncthreads();
        if (threadIdx.x < 16 * MT) {
            const int m = m0 + threadIdx.x;
            if (m < a.M) {
                a.part_keys[(size_t)m * a.n_parts + blockIdx.x] = key_s[threadIdx.x];
                if (a.part_lse) {
                    float2 st = float2{-INFINITY, 0.f};
#pragma unroll
                    for (int c = 0; c < CT; ++c) st = lse_merge(st, lse_s[threadIdx.x][c]);
                    a.part_lse[(size_t)m * a.n_parts + blockIdx.x] = st;
                }
            }
        }
    }
#ifdef NLD_TIMELINE
    __syncthreads();
#endif
    NLD_TS(TL_O, 2);
}

template <int EPI, int MT, bool XK>
static hipError_t launch_stream_ct(int ct, int nw, dim3 grid, const GemmArgs& a, hipStream_t s) {
    if (ct == 1 && nw == 8) launch(gemm_stream_kernel<MT, 1, 8, EPI, XK>, dim3(grid), dim3(512), s, a);
    else if (ct == 1 && nw == 16 && !XK) {
        if constexpr (!XK) launch(gemm_stream_kernel<MT, 1, 16, EPI, false>, dim3(grid), dim3(1024), s, a);
    }
    else if (ct == 2 && nw == 8) launch(gemm_stream_kernel<MT, 2, 8, EPI, XK>, dim3(grid), dim3(512), s, a);
    else if (ct == 4 && nw == 4) launch(gemm_stream_kernel<MT, 4, 4, EPI, XK>, dim3(grid), dim3(256), s, a);
    else if (ct == 1 && nw == 4) launch(gemm_stream_kernel<MT, 1, 4, EPI, XK>, dim3(grid), dim3(256), s, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

template <int EPI, bool XK = false>
static hipError_t launch_stream_mt(int mt, int ct, int nw, dim3 grid, const GemmArgs& a, hipStream_t s) {
    switch (mt) {
        case 1: return launch_stream_ct<EPI, 1, XK>(ct, nw, grid, a, s);
        case 2: return launch_stream_ct<EPI, 2, XK>(ct, nw, grid, a, s);
        case 4: return launch_stream_ct<EPI, 4, XK>(ct, nw, grid, a, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gemm_stream(int epi, int mt, int ct, int nw, int grid_x, int grid_y, const GemmArgs& a,
                              hipStream_t s) {
    const dim3 grid(grid_x, grid_y);
    if (a.W2 && epi != EPI_RESID) return hipErrorInvalidValue;
    switch (epi) {
        case EPI_QKV: return launch_stream_mt<EPI_QKV>(mt, ct, nw, grid, a, s);
        case EPI_RESID:
            return a.W2 ? launch_stream_mt<EPI_RESID, true>(mt, ct, nw, grid, a, s)
                        : launch_stream_mt<EPI_RESID>(mt, ct, nw, grid, a, s);
        case EPI_SWIGLU: return launch_stream_mt<EPI_SWIGLU>(mt, ct, nw, grid, a, s);
        case EPI_LMHEAD: return launch_stream_mt<EPI_LMHEAD>(mt, ct, nw, grid, a, s);
        case EPI_SPLIT: return launch_stream_mt<EPI_SPLIT>(mt, ct, nw, grid, a, s);
        default: return hipErrorInvalidValue;
    }
}

// =====================================================================================
// Split-K GEMM (O and down projections with the residual epilogue, and the normed QKV and
// gate/up projections; M <= 64).  Workgroup (column group cg,
// K slice ks) multiplies its slice of the operand against CT column tiles, so the
// operand is read once per CT tiles and K slice instead of once per tile (the split
// operand is twice as large as the weights it multiplies in these projections).  The
// NW wavefronts cut the slice further and meet in LDS.  With ksplit > 1 the workgroup's
// partial [16*MT rows][16*CT columns] goes to the workspace with agent-scope stores
// (written through to memory, so that every XCD sees them); once every lane's stores
// are acknowledged, one atomic on the group's counter counts the workgroup in.  The
// workgroup that arrives last reads the other partials with agent-scope loads (which
// do not hit stale lines of its own L2), adds the ksplit partials in slice order (the
// sum does not depend on which workgroup is last), sets the counter back to zero for
// the next launch and runs the residual epilogue.  No workgroup ever waits for
// another: there is no spin and no cache-wide fence.
// =====================================================================================
// Operand and weight registers of one batch of the split-K GEMM: U k-steps.
template <int MT, int CT, int U>
struct SkBatch {
    uint4 w[U][CT];
    uint4 x[U][MT];
    uint4 xl[U][MT];
};

template <int MT, int CT, int NW, int EPI>
__global__ void __launch_bounds__(NW * 64) gemm_splitk_kernel(GemmArgs a, float* part, unsigned* ctr, int ksplit) {
    // Up to two row tiles: separate hi and lo accumulators and batches of several k-steps.  Four row
    // tiles: one accumulator per output tile takes both operand halves and a batch is one k-step
    // (the registers of 16 tiles' accumulators and of 12 operand quads per k-step).
    constexpr bool MERGE = MT >= 4;
    constexpr int U = MERGE ? 1 : Batch<MT, CT, true>::U;
    typedef SkBatch<MT, CT, U> B;
    constexpr int NTL = MT * CT;   // output tiles of the workgroup; wavefront w finishes tiles w, w + NW, ...
    constexpr bool NORMED = EPI == EPI_QKV || EPI == EPI_SWIGLU;
    static_assert(EPI == EPI_RESID || NORMED, "residual, QKV or SwiGLU epilogue");
    __shared__ f32x4_t red[NW][NTL][64];
    __shared__ float inv_s[16 * MT];
    __shared__ int last_s;
    // timeline class: a residual projection whose reduction is longer than its output is the down
    // projection, otherwise the O projection
    const int TLC = EPI == EPI_QKV ? TL_QKV : (EPI == EPI_SWIGLU ? TL_GATE_UP : (a.K > a.n_tiles * 16 ? TL_DOWN : TL_O));
    (void)TLC;
    NLD_TS(TLC, 0);

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int cg = blockIdx.x, ks = blockIdx.y;
    const int t0 = cg * CT;
    const int N = a.n_tiles * 16;

    // the workgroup's k-steps [kb, ke), then the wavefront's share [s_begin, s_end)
    const int per_wg = (a.ksteps + ksplit - 1) / ksplit;
    const int kb = min(a.ksteps, ks * per_wg), ke = min(a.ksteps, kb + per_wg);
    const int per = (ke - kb + NW - 1) / NW;
    const int s_begin = min(ke, kb + wave * per);
    const int s_end = min(ke, s_begin + per);

    // epilogue inputs of this wavefront's first tile, fetched up front: residual rows 4g + i
    // of the tile and the next RMSNorm gain of column r
    float xres[4] = {0.f, 0.f, 0.f, 0.f}, gn = 0.f;
    if (EPI == EPI_RESID && wave < NTL) {
        const int mt = wave / CT, t = t0 + wave % CT;
        if (t < a.n_tiles) {
            gn = bf16_to_f32(a.gain_next[t * 16 + r]);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int m = 16 * mt + 4 * g + i;
                if (m < a.M) xres[i] = a.x[(size_t)m * N + t * 16 + r];
            }
        }
    }

    const uint4* wp[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) wp[ct] = a.W + (size_t)min(t0 + ct, a.n_tiles - 1) * a.ksteps * 64 + lane;
    const uint16_t* ap[MT];
    bool aok[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        aok[mt] = mt * 16 + r < a.M;
        ap[mt] = a.A + (size_t)mt * a.ksteps * 1024 + (size_t)lane * 8;
    }

    f32x4_t acc[MT][CT], accl[MERGE ? 1 : MT][MERGE ? 1 : CT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[mt][ct] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if constexpr (!MERGE) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) accl[mt][ct] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }

    const uint4 zero4 = {0u, 0u, 0u, 0u};
    auto load = [&](int s, B& buf) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int ss = s + u;
            const bool in = ss < s_end;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) buf.w[u][ct] = in ? wp[ct][(size_t)ss * 64] : zero4;
            const int kcol = ss * 32 + 8 * g;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const bool ok = in && aok[mt] && kcol < a.K;
                buf.x[u][mt] = ok ? *(const uint4*)(ap[mt] + (size_t)ss * 1024) : zero4;
                buf.xl[u][mt] = ok ? *(const uint4*)(ap[mt] + (size_t)ss * 1024 + SPLIT_LO) : zero4;
            }
        }
    };
    auto compute = [&](const B& buf) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int ct = 0; ct < CT; ++ct) {
                    acc[mt][ct] = mfma_16x16x32(buf.x[u][mt], buf.w[u][ct], acc[mt][ct]);
                    if constexpr (MERGE) acc[mt][ct] = mfma_16x16x32(buf.xl[u][mt], buf.w[u][ct], acc[mt][ct]);
                    else accl[mt][ct] = mfma_16x16x32(buf.xl[u][mt], buf.w[u][ct], accl[mt][ct]);
                }
    };

    B b0, b1;
    load(s_begin, b0);
    if constexpr (NORMED) rms_scales(a, 0, 16 * MT, inv_s);   // visible after the barrier below
    for (int s = s_begin; s < s_end; s += 2 * U) {
        load(s + U, b1);
        compute(b0);
        load(s + 2 * U, b0);
        compute(b1);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            if constexpr (MERGE) red[wave][mt * CT + ct][lane] = acc[mt][ct];
            else red[wave][mt * CT + ct][lane] = acc[mt][ct] + accl[mt][ct];
        }
    __syncthreads();
    NLD_TS(TLC, 1);   // main loop done

    typedef unsigned long long u64;
    // the workgroup's partials of the wavefront's tiles ti = wave, wave + NW, ... (fixed order over
    // the wavefronts), kept in registers and, with ksplit > 1, stored for the last workgroup
    constexpr int TPW = (NTL + NW - 1) / NW;
    f32x4_t v[TPW];
#pragma unroll
    for (int q = 0; q < TPW; ++q) {
        const int ti = wave + q * NW;
        v[q] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        if (ti < NTL) {
#pragma unroll
            for (int w = 0; w < NW; ++w) v[q] += red[w][ti][lane];
        }
    }
    if (ksplit > 1) {
#pragma unroll
        for (int q = 0; q < TPW; ++q) {
            const int ti = wave + q * NW;
            if (ti < NTL) {
                u64* pp = (u64*)(part + ((((size_t)cg * ksplit + ks) * NTL + ti) * 64 + lane) * 4);
                __hip_atomic_store(pp, __builtin_bit_cast(u64, f32x2_t{v[q][0], v[q][1]}), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(pp + 1, __builtin_bit_cast(u64, f32x2_t{v[q][2], v[q][3]}), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        // every lane's stores are acknowledged before the workgroup counts itself in
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_s_waitcnt(0);
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __syncthreads();
        if (threadIdx.x == 0)
            last_s = __hip_atomic_fetch_add(ctr + cg, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (unsigned)(ksplit - 1);
        __syncthreads();
        NLD_TS(TLC, 2);   // partial counted in
        if (!last_s) return;
        if (threadIdx.x == 0) __hip_atomic_exchange(ctr + cg, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int q = 0; q < TPW; ++q) {
            const int ti = wave + q * NW;
            if (ti >= NTL) continue;
            f32x4_t sum = {0.f, 0.f, 0.f, 0.f};
            for (int sl = 0; sl < ksplit; ++sl) {
                if (sl == ks) {
                    sum += v[q];
                    continue;
                }
                const u64* qq = (const u64*)(part + ((((size_t)cg * ksplit + sl) * NTL + ti) * 64 + lane) * 4);
                const f32x2_t lo = __builtin_bit_cast(f32x2_t, __hip_atomic_load(qq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
                const f32x2_t hi = __builtin_bit_cast(f32x2_t, __hip_atomic_load(qq + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
                sum += f32x4_t{lo[0], lo[1], hi[0], hi[1]};
            }
            v[q] = sum;
        }
    }
#pragma unroll
    for (int q = 0; q < TPW; ++q) {
        const int ti = wave + q * NW;
        if (ti >= NTL) continue;
        const int mt = ti / CT, t = t0 + ti % CT;
        if (t >= a.n_tiles) continue;
        if (EPI == EPI_RESID && q > 0) {
            gn = bf16_to_f32(a.gain_next[t * 16 + r]);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int m = 16 * mt + 4 * g + i;
                xres[i] = m < a.M ? a.x[(size_t)m * N + t * 16 + r] : 0.f;
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int m = 16 * mt + 4 * g + i;
            if constexpr (EPI == EPI_RESID) {
                epi_resid(a, v[q][i], m, t, lane, xres[i], gn);
            } else if constexpr (EPI == EPI_QKV) {
                const int mc = min(m, a.M - 1);
                const int pos = committed_length(a.lengths, mc / a.k_blk, a.max_len, a.status) + mc % a.k_blk;
                epi_qkv(a, v[q][i] * inv_s[m], m, t, lane, pos);
            } else {
                epi_swiglu(a, v[q][i] * inv_s[m], m, t, lane);
            }
        }
    }
}

bool gemm_splitk_supported(int epi, int M, int ct) {
    return (epi == EPI_RESID || epi == EPI_QKV || epi == EPI_SWIGLU) && M >= 1 && M <= 64 && ct >= 2 && ct <= 4;
}

template <int EPI, int CT>
static void launch_splitk_ct(dim3 grid, int mt, const GemmArgs& a, float* part, unsigned* ctr, int ksplit,
                             hipStream_t s) {
    if (mt == 4) launch(gemm_splitk_kernel<4, CT, 8, EPI>, grid, dim3(512), s, a, part, ctr, ksplit);
    else if (mt == 2) launch(gemm_splitk_kernel<2, CT, 8, EPI>, grid, dim3(512), s, a, part, ctr, ksplit);
    else launch(gemm_splitk_kernel<1, CT, 8, EPI>, grid, dim3(512), s, a, part, ctr, ksplit);
}

template <int EPI>
static void launch_splitk_epi(int ct, dim3 grid, int mt, const GemmArgs& a, float* part, unsigned* ctr, int ksplit,
                              hipStream_t s) {
    if (ct == 4) launch_splitk_ct<EPI, 4>(grid, mt, a, part, ctr, ksplit, s);
    else if (ct == 3) launch_splitk_ct<EPI, 3>(grid, mt, a, part, ctr, ksplit, s);
    else launch_splitk_ct<EPI, 2>(grid, mt, a, part, ctr, ksplit, s);
}

hipError_t launch_gemm_splitk(int epi, int ct, int ksplit, const GemmArgs& a, float* part, unsigned* ctr,
                              hipStream_t s) {
    if (!gemm_splitk_supported(epi, a.M, ct) || a.W2 || ksplit < 1 || ksplit > SPLITK_MAX) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((a.n_tiles + ct - 1) / ct), (unsigned)ksplit);
    const int mt = a.M > 32 ? 4 : (a.M > 16 ? 2 : 1);
    if (epi == EPI_RESID) launch_splitk_epi<EPI_RESID>(ct, grid, mt, a, part, ctr, ksplit, s);
    else if (epi == EPI_QKV) launch_splitk_epi<EPI_QKV>(ct, grid, mt, a, part, ctr, ksplit, s);
    else launch_splitk_epi<EPI_SWIGLU>(ct, grid, mt, a, part, ctr, ksplit, s);
    return hipGetLastError();
}

// =====================================================================================
// Tiled GEMM for many rows (M > 64), where the projections approach the MFMA ridge: a
// workgroup computes a 128-row x 128-column output tile over the whole reduction, so the
// weights stream once per 128 rows and the operand once per 128 columns.  Per stage of
// two k-steps the operand's eight row tiles (split: hi and lo) and the weights' eight
// column tiles are copied into LDS, double buffered, with the next stage's global loads
// in flight in registers while the current one is multiplied.  Wavefront w multiplies
// row tiles 2(w/2), +1 against column tiles 4(w%2) .. +3 (8 MFMAs per operand half and
// k-step).  Workgroups are ordered so that the row groups sharing a column group run
// next to each other on one XCD (workgroup b runs on XCD b % 8) and find its weight
// tiles in that XCD's L2.  Epilogues as in the other GEMMs.
// =====================================================================================
namespace tile {
constexpr int BR = 8;                        // row tiles per workgroup
constexpr int BC = 8;                        // column tiles per workgroup
constexpr int KS = 1;                        // k-steps per stage
constexpr int A_CHUNKS = BR * KS * 2;        // 1 KiB operand blocks per stage (hi and lo)
constexpr int W_CHUNKS = BC * KS;            // 1 KiB weight blocks per stage
constexpr int CHUNKS = A_CHUNKS + W_CHUNKS;
constexpr int NT = 512;
constexpr int CPT = CHUNKS * 64 / NT;        // 16-byte pieces per thread per stage
constexpr int PD = 4;                        // stages in flight in registers (even: LDS buffer = stage & 1)
static_assert(PD % 2 == 0, "the LDS buffer of a stage is its parity");
static_assert(A_CHUNKS * 64 % NT == 0 && CHUNKS * 64 % NT == 0, "pieces per thread must split by kind");
}  // namespace tile

// K slices: with ksplit > 1, workgroup (x, y) multiplies the y-th of ksplit near-equal runs of
// stages of its 128 x 128 tile and stores its accumulators to `part` with agent-scope stores; the
// workgroup that completes the tile's counter adds the slices in slice order and runs the
// epilogue, then resets the counter.
template <int EPI>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(4)))
gemm_tile_kernel(GemmArgs a, int R, int C, int ksplit, float* part, unsigned* ctr) {
    using namespace tile;
    constexpr bool NORMED = EPI == EPI_QKV || EPI == EPI_SWIGLU || EPI == EPI_LMHEAD;
    __shared__ uint4 lds[2][CHUNKS * 64];
    __shared__ float inv_s[BR * 16];
    __shared__ int pos_s[BR * 16];
    __shared__ unsigned long long key_s[BR * 16];
    __shared__ float2 lse_s[BR * 16][BC];

    const int b = blockIdx.x, xcd = b & 7, gi = b >> 3;
    const int rg = gi % R, c = (gi / R) * 8 + xcd;
    if (c >= C) return;   // the whole workgroup leaves: the grid covers whole groups of 8 column groups
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int wr = wave >> 1, wc = wave & 1;
    const int m0 = rg * BR * 16;

    if constexpr (EPI == EPI_LMHEAD) {
        if (threadIdx.x < BR * 16) {
            key_s[threadIdx.x] = 0ull;
#pragma unroll
            for (int j = 0; j < BC; ++j) lse_s[threadIdx.x][j] = float2{-INFINITY, 0.f};
        }
    }
    if constexpr (NORMED) rms_scales(a, m0, BR * 16, inv_s);
    if constexpr (EPI == EPI_QKV) {
        if (threadIdx.x < BR * 16) {
            const int m = min(m0 + (int)threadIdx.x, a.M - 1);
            pos_s[threadIdx.x] = committed_length(a.lengths, m / a.k_blk, a.max_len, a.status) + m % a.k_blk;
        }
    }

    // Stage pieces: thread (wave, lane) copies piece q = 1 KiB block wave + 8q, 16 bytes at
    // lane.  Blocks 0 .. A_CHUNKS-1 are operand blocks (row tile, k-step, half), the rest
    // weight blocks (column tile, k-step).  The launcher guarantees whole stages (ksteps a
    // multiple of KS, K a multiple of 32) and operand rows allocated up to a multiple of
    // 128; column tiles past the end are read clamped and their outputs dropped.  So every
    // load is unconditional and in bounds.
    static_assert(A_CHUNKS % 8 == 0 && CHUNKS == 8 * CPT, "8 blocks per piece index");
    // slice ksl: stages [ksl*n/ksplit, (ksl+1)*n/ksplit), at least one since ksplit <= n
    const int ksl = blockIdx.y;
    const int nst_all = a.ksteps / KS;
    const int st0 = ksl * nst_all / ksplit;
    const int nst = (ksl + 1) * nst_all / ksplit - st0;
    const uint4* srcp[CPT];   // stage 0 address of each piece (the slice's first stage)
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
        const int chunk = wave + 8 * q;
        if (q < A_CHUNKS / 8) {
            const int rt = chunk / (KS * 2), ks = (chunk / 2) % KS, half = chunk & 1;
            srcp[q] = (const uint4*)(a.A + ((size_t)((m0 / 16 + rt) * a.ksteps + ks) * 2 + half) * 512) + lane;
        } else {
            const int wck = chunk - A_CHUNKS, ct = wck / KS, ks = wck % KS;
            srcp[q] = a.W + ((size_t)min(c * BC + ct, a.n_tiles - 1) * a.ksteps + ks) * 64 + lane;
        }
        srcp[q] += (size_t)st0 * KS * (q < A_CHUNKS / 8 ? 128 : 64);
    }
    // stage st: operand blocks advance by KS k-steps of 2 KiB, weight blocks by KS of 1 KiB
    typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
#define NLD_TILE_GLOAD(st, dst)                                                            \
    _Pragma("unroll") for (int q = 0; q < CPT; ++q)                                         \
        dst[q] = *(const u32x4_t*)(srcp[q] + (size_t)(st) * KS * (q < A_CHUNKS / 8 ? 128 : 64))
#define NLD_TILE_LSTORE(v, buf) \
    _Pragma("unroll") for (int q = 0; q < CPT; ++q) *(u32x4_t*)&lds[buf][threadIdx.x + q * NT] = v[q]

    // one accumulator per output tile takes both operand halves (eight independent tiles keep
    // the MFMA pipeline busy between the two dependent products)
    f32x4_t acc[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    auto compute = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            uint4 ah[2], al[2], w[4];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int rt = 2 * wr + i;
                ah[i] = lds[buf][((rt * KS + ks) * 2 + 0) * 64 + lane];
                al[i] = lds[buf][((rt * KS + ks) * 2 + 1) * 64 + lane];
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) w[j] = lds[buf][(A_CHUNKS + (4 * wc + j) * KS + ks) * 64 + lane];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = mfma_16x16x32(ah[i], w[j], acc[i][j]);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = mfma_16x16x32(al[i], w[j], acc[i][j]);
        }
    };

    // Stage s is multiplied from LDS buffer s & 1 while stages s+1 .. s+PD wait or are in flight in
    // a ring of PD register slots: the slot of stage s is refilled with stage s+PD as soon as s is
    // in LDS, so PD stages of loads cover the L2 / HBM latency.  The loop is unrolled by PD so
    // that every slot index is a compile-time constant; loads past the last stage re-read it and
    // are never stored.
    u32x4_t rb[PD][CPT];
#pragma unroll
    for (int p = 0; p < PD; ++p) NLD_TILE_GLOAD(min(p, nst - 1), rb[p]);
    NLD_TILE_LSTORE(rb[0], 0);
    __syncthreads();
    for (int st = 0; st < nst; st += PD) {
#pragma unroll
        for (int u = 0; u < PD; ++u) {
            const int cur = st + u;
            if (cur >= nst) break;
            NLD_TILE_GLOAD(min(cur + PD, nst - 1), rb[u]);
            compute(u & 1);
            if (cur + 1 < nst) { NLD_TILE_LSTORE(rb[(u + 1) % PD], (u + 1) & 1); }
            __syncthreads();
        }
    }
#undef NLD_TILE_GLOAD
#undef NLD_TILE_LSTORE

    if (ksplit > 1) {
        // slice partials, 16 pairs of floats per thread, pair-major so that every store is one
        // contiguous 512-byte run per wavefront
        typedef unsigned long long u64;
        __shared__ int last_s;
        const int grp = c * R + rg;
        u64* pp = (u64*)part + (size_t)(grp * ksplit + ksl) * 16 * NT + threadIdx.x;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int q = (i * 4 + j) * 2;
                __hip_atomic_store(pp + (size_t)q * NT, __builtin_bit_cast(u64, f32x2_t{acc[i][j][0], acc[i][j][1]}),
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(pp + (size_t)(q + 1) * NT, __builtin_bit_cast(u64, f32x2_t{acc[i][j][2], acc[i][j][3]}),
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        // every lane's stores are acknowledged before the workgroup counts itself in
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_s_waitcnt(0);
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __syncthreads();
        if (threadIdx.x == 0)
            last_s = __hip_atomic_fetch_add(ctr + grp, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (unsigned)(ksplit - 1);
        __syncthreads();
        if (!last_s) return;
        if (threadIdx.x == 0) __hip_atomic_exchange(ctr + grp, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        f32x4_t sum[2][4];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) sum[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int sl = 0; sl < ksplit; ++sl) {   // fixed order over the slices
            if (sl == ksl) {
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) sum[i][j] += acc[i][j];
                continue;
            }
            const u64* qq = (const u64*)part + (size_t)(grp * ksplit + sl) * 16 * NT + threadIdx.x;
            f32x2_t v[16];
#pragma unroll
            for (int q = 0; q < 16; ++q)
                v[q] = __builtin_bit_cast(f32x2_t, __hip_atomic_load(qq + (size_t)q * NT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int q = (i * 4 + j) * 2;
                    sum[i][j] += f32x4_t{v[q][0], v[q][1], v[q + 1][0], v[q + 1][1]};
                }
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = sum[i][j];
    }

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const f32x4_t v = acc[i][j];
            const int rt = 2 * wr + i, ct = 4 * wc + j;
            const int t = c * BC + ct;
            if (t >= a.n_tiles) continue;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int ml = rt * 16 + 4 * g + e;
                const int m = m0 + ml;
                if constexpr (EPI == EPI_RESID) {
                    const int N = a.n_tiles * 16;
                    const float xr = m < a.M ? a.x[(size_t)m * N + t * 16 + r] : 0.f;
                    epi_resid(a, v[e], m, t, lane, xr, bf16_to_f32(a.gain_next[t * 16 + r]));
                } else if constexpr (EPI == EPI_QKV) {
                    epi_qkv(a, v[e] * inv_s[ml], m, t, lane, pos_s[ml]);
                } else if constexpr (EPI == EPI_SWIGLU) {
                    epi_swiglu(a, v[e] * inv_s[ml], m, t, lane);
                } else {
                    float2 tl;
                    const unsigned long long key = epi_lmhead(a, v[e] * inv_s[ml], m, t, lane, &tl);
                    if (r == 0) {
                        atomicMax(&key_s[ml], key);
                        if (a.part_lse) lse_s[ml][ct] = tl;   // each (row, column tile) is finished once
                    }
                }
            }
        }
    if constexpr (EPI == EPI_LMHEAD) {
        __syncthreads();
        if (threadIdx.x < BR * 16) {
            const int m = m0 + threadIdx.x;
            if (m < a.M) {
                a.part_keys[(size_t)m * a.n_parts + c] = key_s[threadIdx.x];
                if (a.part_lse) {
                    float2 st = float2{-INFINITY, 0.f};
#pragma unroll
                    for (int j = 0; j < BC; ++j) st = lse_merge(st, lse_s[threadIdx.x][j]);
                    a.part_lse[(size_t)m * a.n_parts + c] = st;
                }
            }
        }
    }
}

int gemm_tile_parts(int n_tiles) { return (n_tiles + tile::BC - 1) / tile::BC; }

bool gemm_tile_supported(int M, int K, int ksteps) {
    return M > 64 && K % 32 == 0 && ksteps % tile::KS == 0 && ksteps >= tile::KS;
}

int gemm_tile_row_pad() { return tile::BR * 16; }

int gemm_tile_groups(int M, int n_tiles) { return ((M + tile::BR * 16 - 1) / (tile::BR * 16)) * gemm_tile_parts(n_tiles); }
int gemm_tile_stages(int ksteps) { return ksteps / tile::KS; }
size_t gemm_tile_part_floats_per_wg() { return (size_t)tile::NT * 32; }
int gemm_tile_wgs_per_cu() { return 2; }

hipError_t launch_gemm_tile(int epi, const GemmArgs& a, int ksplit, float* part, unsigned* ctr, hipStream_t s) {
    if (!gemm_tile_supported(a.M, a.K, a.ksteps) || a.W2) return hipErrorInvalidValue;
    // every slice gets at least one stage; the LM head's argmax partials are per column group
    if (ksplit < 1 || ksplit > gemm_tile_stages(a.ksteps) || (ksplit > 1 && (!part || !ctr || epi == EPI_LMHEAD)))
        return hipErrorInvalidValue;
    const int R = (a.M + tile::BR * 16 - 1) / (tile::BR * 16);
    const int C = gemm_tile_parts(a.n_tiles);
    const dim3 grid((unsigned)(R * ((C + 7) / 8) * 8), (unsigned)ksplit), blk(tile::NT);
    switch (epi) {
        case EPI_QKV: launch(gemm_tile_kernel<EPI_QKV>, grid, blk, s, a, R, C, ksplit, part, ctr); break;
        case EPI_RESID: launch(gemm_tile_kernel<EPI_RESID>, grid, blk, s, a, R, C, ksplit, part, ctr); break;
        case EPI_SWIGLU: launch(gemm_tile_kernel<EPI_SWIGLU>, grid, blk, s, a, R, C, ksplit, part, ctr); break;
        case EPI_LMHEAD: launch(gemm_tile_kernel<EPI_LMHEAD>, grid, blk, s, a, R, C, ksplit, part, ctr); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// =====================================================================================
// Block-masked GQA attention.  Workgroup = (key split, sequence x KV head, row slice);
// one compute wavefront per 16 query rows of the GQA group (rows = heads of the
// group x block rows).  The committed prefix [0, P) is cut into key splits that
// read the bf16 cache; one more workgroup per (unit, row slice), the block part,
// covers the block's own k keys (causal or bidirectional per the mode) from the
// split K/V the QKV epilogue left in the workspace, so this pass sees its own keys
// and values at about 16 significant bits while the cache keeps bf16.  Keys stream
// through LDS in stages of 64 (K rows and the transposed V tile, XOR-swizzled for
// conflict-free operand reads), double buffered: the next stage's global loads are
// in flight while the current one is multiplied.  S^T = K Q^T on MFMA puts one
// query row per lane column, so a row's softmax statistics live in lanes r, r+16,
// r+32, r+48 and P^T is already the B operand of O^T = V^T P^T.  Queries and P are
// split operands.  Online softmax in base 2, fp32; every workgroup writes one
// partial (max, sum, unnormalised output) per row for the merge.
// =====================================================================================
template <int D>
struct AttnCfg {
    static constexpr int KCH = D / 8;                    // 16-byte chunks per K row
    static constexpr int KCHUNKS = 64 * KCH;             // K tile chunks per stage
    static constexpr int VCHUNKS = D * 8;                // V tile chunks per stage (D rows x 64 keys)
    static constexpr int CHUNKS = KCHUNKS + VCHUNKS;
};

// XOR swizzles (chunk index within a row): make the 16 rows read by one MFMA
// operand load hit 16 distinct bank groups.
template <int D>
__device__ __forceinline__ int kswz(int row) {
    if constexpr (D == 128) return (row & 3) | ((row >> 1) & 12);
    else return ((row >> 1) & 1) | ((row >> 2) & 6);
}
__device__ __forceinline__ int vswz(int d) { return (d >> 1) & 7; }

// key of S-tile tau, tile row rho within a 64-key stage: the eight keys a lane group
// holds for one PV k-step are then consecutive.
__device__ __forceinline__ int stage_key(int tau, int rho) {
    return 32 * (tau >> 1) + 8 * (rho >> 2) + 4 * (tau & 1) + (rho & 3);
}

// committed length of sequence b as the attention reads it: clamped to [0, max_len]
__device__ __forceinline__ int attn_length(const AttnArgs& a, int b) {
    const int p = a.lengths[b];
    return p < 0 ? 0 : (p > a.max_len ? a.max_len : p);
}

// Length-aware work item `item` -> (unit, split), split == n_splits for the block part; false past
// the last item.  Wavefront 0 scans the sequences' item counts (nkv * (ceil(P_b / chunk) + 1)) 64
// at a time; the result goes to every thread through LDS.
__device__ bool attn_item(const AttnArgs& a, int item, int* unit, int* split) {
    __shared__ int su_s, ss_s;
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        int base = 0, su = -1, ss = 0;
        for (int b0 = 0; b0 < a.n_seq && su < 0; b0 += 64) {
            const int b = b0 + lane;
            const int nc = b < a.n_seq ? (attn_length(a, b) + a.chunk - 1) / a.chunk : 0;
            const int cnt = b < a.n_seq ? (nc + 1) * a.n_kv_heads : 0;
            int incl = cnt;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const int t = __shfl_up(incl, off);
                if (lane >= off) incl += t;
            }
            const int excl = incl - cnt;
            const bool mine = cnt > 0 && item >= base + excl && item < base + incl;
            const unsigned long long who = __ballot(mine);
            if (who) {
                const int src = __ffsll((long long)who) - 1;
                const int r = __shfl(item - base - excl, src), ncs = __shfl(nc, src);
                su = (b0 + src) * a.n_kv_heads + r / (ncs + 1);
                ss = r % (ncs + 1) == ncs ? a.n_splits : r % (ncs + 1);
            }
            base += __shfl(incl, 63);
        }
        if (lane == 0) {
            su_s = su;
            ss_s = ss;
        }
    }
    __syncthreads();
    *unit = su_s;
    *split = ss_s;
    return su_s >= 0;
}

template <int D, int KH>
__global__ void __launch_bounds__(512) attention_kernel(AttnArgs a) {
    typedef AttnCfg<D> C;
    constexpr int DC = D / 32;
    constexpr int DT = D / 16;
    constexpr int NT = 512;                    // threads per workgroup
    constexpr int CPT = C::CHUNKS / NT;        // stage chunks per thread
    constexpr int RZ = 8 / KH;                 // row tiles per workgroup
    constexpr int TPW = 4 / KH;                // S tiles (16 keys) per wavefront per stage
    constexpr float RESCALE_SLACK = 8.0f;      // log2 headroom before the reference max moves
    // two stage slots, each K tile (KCHUNKS) followed by the V tile (VCHUNKS)
    __shared__ uint4 lds[2 * C::CHUNKS];

    NLD_TS(TL_ATTENTION, 0);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    int split = blockIdx.x, unit = blockIdx.y;
    if (a.items && !attn_item(a, blockIdx.x, &unit, &split)) return;   // the whole workgroup leaves
    const bool blockpart = split == a.n_splits;   // the block's own keys, read in split form
    const int nkv = a.n_kv_heads, G = a.n_q_heads / nkv;
    const int b = unit / nkv, kvh = unit % nkv;
    const int k = a.k_blk, R = G * k;
    const int kh = wave / RZ;                  // which half of each stage's keys (KH == 2)
    const int rt = blockIdx.z * RZ + (wave % RZ);
    const bool computes = rt < a.row_tiles;
    const int row = rt * 16 + r;
    const bool row_ok = computes && row < R;
    const int j = row_ok ? row % k : 0;

    const int P_raw = a.lengths[b];   // requested first; the loads below do not depend on it
    // Block columns this row sees.  Verify: c <= j.  Draft: every column from row bidir_from on.
    // Quadratic layout (mode 2, chain length qk): chain row j sees chain columns c <= j; a mask of
    // group grp sees chain columns c <= grp and the columns [lo_c, hi_c) of its own group.
    const int qk = a.quad_k;
    const bool quad = a.mode == 2;
    const bool bidir_row = (a.mode == 1) && (j >= a.bidir_from);
    const int grp = (quad && j >= qk) ? (j - qk) / qk : j;
    const int lo_c = (quad && j >= qk) ? qk + grp * qk : k, hi_c = (quad && j >= qk) ? lo_c + qk : k;
    int split_beg = split * a.chunk;   // prefix splits: first key of the split (< max_len)

    const size_t head_off = (size_t)(b * nkv + kvh) * a.max_len * D;
    const uint16_t* kbase = a.kc + head_off;   // where gload reads stages from
    const uint16_t* vbase = a.vc + head_off;

    // per-thread stage chunks: global offsets within a stage and LDS slots (swizzled)
    int goff[CPT], loff[CPT];
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
        const int q = threadIdx.x + i * NT;
        if (q < C::KCHUNKS) {
            const int kr = q / C::KCH, c = q % C::KCH;
            goff[i] = q * 8;                                   // relative to kbase + kb * D
            loff[i] = kr * C::KCH + (c ^ kswz<D>(kr));
        } else {
            const int qv = q - C::KCHUNKS, d = qv >> 3, c = qv & 7;
            goff[i] = qv * 8;                                  // relative to the V tile
            loff[i] = C::KCHUNKS + d * 8 + (c ^ vswz(d));      // V slots follow the K slots
        }
    }
    struct Stage {
        uint4 v[CPT];
    };
    auto gload = [&](int kb) __attribute__((always_inline)) {
        Stage st;
        const uint16_t* kp = kbase + (size_t)kb * D;
        const uint16_t* vp = vbase + (size_t)(kb >> 6) * D * 64;
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const bool is_k = threadIdx.x + i * NT < C::KCHUNKS;   // resolved at compile time for most i
            st.v[i] = *(const uint4*)((is_k ? kp : vp) + goff[i]);
        }
        return st;
    };
    auto lstore = [&](const Stage& st, int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) lds[buf * C::CHUNKS + loff[i]] = st.v[i];
    };

    // operand offsets in LDS (per lane, fixed for every stage)
    int koff[TPW][DC], voff[TPW / 2][DT];
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
        const int kr = stage_key(TPW * kh + tt, r);
#pragma unroll
        for (int c = 0; c < DC; ++c) koff[tt][c] = kr * C::KCH + ((4 * c + g) ^ kswz<D>(kr));
    }
#pragma unroll
    for (int kk = 0; kk < TPW / 2; ++kk) {
        const int ks = (TPW / 2) * kh + kk;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const int d = 16 * dt + r;
            voff[kk][dt] = d * 8 + ((4 * ks + g) ^ vswz(d));
        }
    }

    const uint4 zero4 = {0u, 0u, 0u, 0u};
    uint4 qb[DC], ql[DC];   // split queries: hi and lo operands
    {
        const uint16_t* qp = a.q + ((size_t)((unit * a.row_tiles + rt) * DC * 2) * 64 + lane) * 8;
#pragma unroll
        for (int c = 0; c < DC; ++c) {
            qb[c] = row_ok ? *(const uint4*)(qp + (size_t)c * 1024) : zero4;
            ql[c] = row_ok ? *(const uint4*)(qp + (size_t)c * 1024 + SPLIT_LO) : zero4;
        }
    }
    // The first stage is requested before the committed length is known: a prefix split's
    // first 64 keys (always inside the cache; masked below if they are not committed), or
    // the block part's hi and lo halves.
    Stage s0{}, s1{}, s2{};
    if (blockpart) {
        const size_t kv_unit = (size_t)unit * 2 * 64 * D;
        kbase = a.blk_k + kv_unit;
        vbase = a.blk_v + kv_unit;
        s0 = gload(0);
        kbase += 64 * D;
        vbase += 64 * D;
        s1 = gload(0);
    } else {
        s0 = gload(split_beg);
    }

    int P = P_raw < 0 ? 0 : (P_raw > a.max_len ? a.max_len : P_raw);
    // One sequence: the n_splits prefix splits are cut from the committed length, chunk =
    // ceil(P / n_splits) rounded up to whole stages (at most the plan's chunk, which was cut from
    // max_len), so that a cache much longer than its prefix still spreads the prefix over every
    // split.  The first stage went out at the plan's split start; it is requested again where
    // the two differ.
    int chunk = a.chunk;
    if (!a.items && !blockpart) {
        chunk = max(64, ((P + a.n_splits - 1) / a.n_splits + 63) / 64 * 64);
        const int beg = split * chunk;
        if (beg != split_beg) {
            split_beg = beg;
            if (beg < P) s0 = gload(beg);   // beg < P <= max_len, a multiple of 64: inside the cache
        }
    }
    // prefix splits cover committed keys [kbeg, kend) of [0, P); the block part covers [P, P + k)
    const int kbeg = blockpart ? P : split_beg;
    const int kend = blockpart ? P + k : min(kbeg + chunk, P);
    const int nst = blockpart ? 1 : (kend > kbeg ? (kend - kbeg + 63) / 64 : 0);
    NLD_TS(TL_ATTENTION, 1);   // committed length known
    if (!blockpart) {
        if (nst > 1 && a.late < 2) s1 = gload(kbeg + 64);
        if (nst > 2 && a.late < 1) s2 = gload(kbeg + 128);
    }

    f32x4_t acc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // p = exp2(s - m_ref): m_ref only moves when a score exceeds it by RESCALE_SLACK,
    // so the accumulators are rescaled rarely (any reference gives the same ratio).
    float m_ref = -INFINITY, l_part = 0.f;

    // kb: first key of the stage.  lo_slot: the block part keeps the lo halves of
    // the block's keys and values in the second stage slot.
    auto compute = [&](int kb, int buf, bool lo_slot) __attribute__((always_inline)) {
        if (!computes) return;
        f32x4_t s[TPW], sl[TPW];
#pragma unroll
        for (int tt = 0; tt < TPW; ++tt) {
            s[tt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            sl[tt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < DC; ++c) {
                const uint4 kop = lds[buf * C::CHUNKS + koff[tt][c]];
                s[tt] = mfma_16x16x32(kop, qb[c], s[tt]);
                sl[tt] = mfma_16x16x32(kop, ql[c], sl[tt]);
                if (lo_slot) sl[tt] = mfma_16x16x32(lds[C::CHUNKS + koff[tt][c]], qb[c], sl[tt]);
            }
            s[tt] += sl[tt];
        }
        const bool edge = (kb + 64 > P) || (kb + 64 > kend);   // stage touches the block or the split end
        float sv[4 * TPW];
        float mloc = -INFINITY;
#pragma unroll
        for (int tt = 0; tt < TPW; ++tt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float x = s[tt][i] * a.scale_log2;
                if (edge) {
                    const int key = kb + stage_key(TPW * kh + tt, 4 * g + i);
                    const int c = key - P;   // block column (keys < P are the prefix)
                    const bool vis = key < kend && (key < P || (quad ? ((c < qk && c <= grp) || (c >= lo_c && c < hi_c))
                                                                     : (c <= j || bidir_row)));
                    x = vis ? x : -INFINITY;
                }
                sv[tt * 4 + i] = x;
                mloc = fmaxf(mloc, x);
            }
        mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
        if (mloc > m_ref + RESCALE_SLACK) {        // new reference: rescale what has accumulated
            const float alpha = __builtin_amdgcn_exp2f(m_ref - mloc);   // 0 when m_ref = -inf
            l_part *= alpha;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) acc[dt] *= alpha;
            m_ref = mloc;
        }
        float p[4 * TPW];
        float psum = 0.f;
#pragma unroll
        for (int e = 0; e < 4 * TPW; ++e) {
            p[e] = __builtin_amdgcn_exp2f(sv[e] - m_ref);   // -inf - finite -> 0; m_ref finite once any key is visible
            psum += p[e];
        }
        if (m_ref == -INFINITY) psum = 0.f;
        l_part += psum;
#pragma unroll
        for (int kk = 0; kk < TPW / 2; ++kk) {
            const int ks = (TPW / 2) * kh + kk;          // 32-key PV step within the stage
            // slot jj of lane group g <-> key kb + 32ks + 8g + jj
            uint4 pop, pol;                               // P^T as split operands
            split8(p + 8 * kk, pop, pol, a.plain & SITE_P);
            if (m_ref == -INFINITY) pop = pol = zero4;
            const int key0 = kb + 32 * ks + 8 * g;
            const bool vmask = edge && (key0 + 8 > kend);  // V rows past the valid keys may hold anything
            auto masked = [&](uint4 vop) __attribute__((always_inline)) {
                if (!vmask) return vop;
                uint32_t w[4] = {vop.x, vop.y, vop.z, vop.w};
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    w[e] = (key0 + 2 * e < kend ? (w[e] & 0xFFFFu) : 0u) | (key0 + 2 * e + 1 < kend ? (w[e] & 0xFFFF0000u) : 0u);
                return uint4{w[0], w[1], w[2], w[3]};
            };
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const uint4 vop = masked(lds[buf * C::CHUNKS + C::KCHUNKS + voff[kk][dt]]);
                acc[dt] = mfma_16x16x32(vop, pop, acc[dt]);
                acc[dt] = mfma_16x16x32(vop, pol, acc[dt]);
                if (lo_slot) acc[dt] = mfma_16x16x32(masked(lds[C::CHUNKS + C::KCHUNKS + voff[kk][dt]]), pop, acc[dt]);
            }
        }
    };

    if (blockpart) {
        // one stage (k <= 64): hi halves in slot 0, lo halves in slot 1
        lstore(s0, 0);
        lstore(s1, 1);
        __syncthreads();
        compute(kbeg, 0, true);
        __syncthreads();
    } else {
        // Stages of 64 keys.  Stage st is multiplied from LDS slot st & 1 while stages st+1
        // and st+2 are in flight in registers (s1 and s2 by turns; the loop is unrolled by
        // two so that no register copy waits on a load still in flight).
        if (nst > 0) lstore(s0, 0);
        if (nst > 1 && a.late >= 2) s1 = gload(kbeg + 64);
        if (nst > 2 && a.late >= 1) s2 = gload(kbeg + 128);
        __syncthreads();
        NLD_TS(TL_ATTENTION, 2);   // first stage in LDS
        for (int st = 0; st < nst; st += 2) {
            compute(kbeg + 64 * st, 0, false);
            if (st + 1 < nst) lstore(s1, 1);
            if (st + 3 < nst) s1 = gload(kbeg + 64 * (st + 3));
            __syncthreads();
            if (st + 1 >= nst) break;
            compute(kbeg + 64 * (st + 1), 1, false);
            if (st + 2 < nst) lstore(s2, 0);
            if (st + 4 < nst) s2 = gload(kbeg + 64 * (st + 4));
            __syncthreads();
        }
    }

    NLD_TS(TL_ATTENTION, 3);   // stages done
    float l_tot = l_part + __shfl_xor(l_part, 16);
    l_tot += __shfl_xor(l_tot, 32);
    if constexpr (KH == 2) {
        // merge the two key halves of each row tile through LDS (the stage buffers are free now)
        float* mrg = (float*)lds;                    // [RZ][16 rows][D + 2] floats, within the 2 stage slots
        float* slot = mrg + ((size_t)(wave % RZ) * 16 + r) * (D + 2);
        if (kh == 1 && computes) {
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int i = 0; i < 4; ++i) slot[16 * dt + 4 * g + i] = acc[dt][i];
            if (g == 0) {
                slot[D] = m_ref;
                slot[D + 1] = l_tot;
            }
        }
        __syncthreads();
        if (kh == 1 || !computes) return;
        const float m2 = slot[D], l2 = slot[D + 1];
        const float mm = fmaxf(m_ref, m2);
        const float w1 = (m_ref == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_ref - mm);
        const float w2 = (m2 == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m2 - mm);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[dt][i] = acc[dt][i] * w1 + slot[16 * dt + 4 * g + i] * w2;
        l_tot = l_tot * w1 + l2 * w2;
        m_ref = mm;
    }
    if (!computes) return;
    const size_t pbase = ((size_t)unit * a.n_parts + split) * a.rows_pad + row;
    float* po = a.part_o + pbase * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) *(float4*)(po + 16 * dt + 4 * g) = float4{acc[dt][0], acc[dt][1], acc[dt][2], acc[dt][3]};
    if (g == 0) *(float2*)(a.part_ml + pbase * 2) = float2{m_ref, l_tot};
#ifdef NLD_TIMELINE
    __syncthreads();
#endif
    NLD_TS(TL_ATTENTION, 4);
}

// Merge of the partials (prefix splits + block part): one workgroup per (unit, query
// row), one thread per head dim; writes the split attention output.
template <int D>
__global__ void __launch_bounds__(D) attention_combine_kernel(AttnArgs a) {
    __shared__ float wsh[256];
    __shared__ float inv_den;
    NLD_TS(TL_COMBINE, 0);
    const int unit = blockIdx.x, rw = blockIdx.y, d = threadIdx.x;
    const int nkv = a.n_kv_heads, G = a.n_q_heads / nkv;
    const int b = unit / nkv, kvh = unit % nkv, k = a.k_blk;
    // parts: prefix splits 0 .. nvalid-1 (the ones holding committed keys), then the block part
    const int nvalid = a.items ? (attn_length(a, b) + a.chunk - 1) / a.chunk : a.n_splits;
    const int ns = nvalid + 1;
    auto pidx = [&](int j) { return j < nvalid ? j : a.n_splits; };
    const size_t ubase = (size_t)unit * a.n_parts * a.rows_pad + rw;
    // With at most FAST parts every load of the workgroup is issued at once: thread d's part
    // statistics and its column of every part's output.  More parts take the looped path.
    constexpr int FAST = 32;
    const bool fast = ns <= FAST;
    float2 ml0 = float2{-INFINITY, 0.f};
    float os[FAST];
    if (fast) {
        if (d < ns) ml0 = *(const float2*)(a.part_ml + (ubase + (size_t)pidx(d) * a.rows_pad) * 2);
#pragma unroll
        for (int e = 0; e < FAST; ++e)
            os[e] = e < ns ? a.part_o[(ubase + (size_t)pidx(e) * a.rows_pad) * D + d] : 0.f;
    }
    // split statistics -> weights exp2(m_s - max) in LDS (ns <= 256)
    float ms = -INFINITY, ls = 0.f;
    if (fast) {
        if (d < ns) wsh[d] = ml0.x;
        ms = ml0.x;
    } else {
        for (int sp = d; sp < ns; sp += D) {
            const float2 ml = *(const float2*)(a.part_ml + (ubase + (size_t)pidx(sp) * a.rows_pad) * 2);
            wsh[sp] = ml.x;
            ms = fmaxf(ms, ml.x);
        }
    }
    // block max over D threads (D <= 128: two wavefronts at most)
    ms = fmaxf(ms, __shfl_xor(ms, 32));
    ms = fmaxf(ms, __shfl_xor(ms, 16));
    ms = fmaxf(ms, __shfl_xor(ms, 8));
    ms = fmaxf(ms, __shfl_xor(ms, 4));
    ms = fmaxf(ms, __shfl_xor(ms, 2));
    ms = fmaxf(ms, __shfl_xor(ms, 1));
    __shared__ float wmax[2];
    if ((d & 63) == 0) wmax[d >> 6] = ms;
    __syncthreads();
    const float mx = (D > 64) ? fmaxf(wmax[0], wmax[1]) : wmax[0];
    if (fast) {
        if (d < ns) {
            const float w = (ml0.x == -INFINITY) ? 0.f : exp2f(ml0.x - mx);
            ls = w * ml0.y;
            wsh[d] = w;
        }
    } else {
        for (int sp = d; sp < ns; sp += D) {
            const float msp = wsh[sp];
            const float w = (msp == -INFINITY) ? 0.f : exp2f(msp - mx);
            ls += w * a.part_ml[(ubase + (size_t)pidx(sp) * a.rows_pad) * 2 + 1];
            wsh[sp] = w;
        }
    }
    ls += __shfl_xor(ls, 32);
    ls += __shfl_xor(ls, 16);
    ls += __shfl_xor(ls, 8);
    ls += __shfl_xor(ls, 4);
    ls += __shfl_xor(ls, 2);
    ls += __shfl_xor(ls, 1);
    __shared__ float wden[2];
    if ((d & 63) == 0) wden[d >> 6] = ls;
    __syncthreads();
    if (d == 0) inv_den = 1.0f / ((D > 64) ? (wden[0] + wden[1]) : wden[0]);
    __syncthreads();
    // the parts in order, one product-sum each (the same order on both paths)
    float num = 0.f;
    if (fast) {
#pragma unroll
        for (int e = 0; e < FAST; ++e)
            if (e < ns) num += wsh[e] * os[e];
    } else {
        int sp = 0;
        for (; sp + 8 <= ns; sp += 8) {
            float o8[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) o8[e] = a.part_o[(ubase + (size_t)pidx(sp + e) * a.rows_pad) * D + d];
#pragma unroll
            for (int e = 0; e < 8; ++e) num += wsh[sp + e] * o8[e];
        }
        for (; sp < ns; ++sp) num += wsh[sp] * a.part_o[(ubase + (size_t)pidx(sp) * a.rows_pad) * D + d];
    }
    const int hl = rw / k, j = rw % k;
    store_split(a.o, split_index(b * k + j, (kvh * G + hl) * D + d, a.n_q_heads * D / 32), num * inv_den,
                a.plain & SITE_O);
    NLD_TS(TL_COMBINE, 1);
}

hipError_t launch_attention(int head_dim, int kh, int zslices, int units, const AttnArgs& a, hipStream_t s) {
    // prefix splits + the block part per unit; length-aware items: all of them on x
    const dim3 grid = a.items ? dim3((a.n_splits + 1) * units, 1, zslices) : dim3(a.n_splits + 1, units, zslices);
    if (head_dim == 128 && kh == 2) launch(attention_kernel<128, 2>, dim3(grid), dim3(512), s, a);
    else if (head_dim == 128 && kh == 1) launch(attention_kernel<128, 1>, dim3(grid), dim3(512), s, a);
    else if (head_dim == 64 && kh == 2) launch(attention_kernel<64, 2>, dim3(grid), dim3(512), s, a);
    else if (head_dim == 64 && kh == 1) launch(attention_kernel<64, 1>, dim3(grid), dim3(512), s, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_attention_combine(int head_dim, int units, int rows, const AttnArgs& a, hipStream_t s) {
    const dim3 grid(units, rows);
    if (head_dim == 128) launch(attention_combine_kernel<128>, dim3(grid), dim3(128), s, a);
    else if (head_dim == 64) launch(attention_combine_kernel<64>, dim3(grid), dim3(64), s, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

// =====================================================================================
// Embedding gather of the block (block assembly per call kind) into the fp32 residual.
// =====================================================================================
__global__ void __launch_bounds__(256) embed_kernel(EmbedArgs a) {
    const int m = blockIdx.x;
    const int b = m / a.k_blk, j = m % a.k_blk;
    if (m == 0)
        for (int i = threadIdx.x; i < a.n_tile_ctr; i += blockDim.x) a.tile_ctr[i] = 0u;
    // RoPE table of this row (used by every layer's QKV epilogue): angle pos * theta_i
    // reduced to [-pi, pi] and evaluated in fp64, stored as fp32 (cos, sin).
    if ((int)threadIdx.x < a.head_dim / 2) {
        const int fi = threadIdx.x;
        // quadratic layout: mask r of group c (row qk + c*qk + r - 1) sits at P + c + r
        const int qk = a.quad_k;
        const int off = (qk > 0 && j >= qk) ? (j - qk) / qk + (j - qk) % qk + 1 : j;
        const int pos = committed_length(a.lengths, b, a.max_len, a.status) + off;
        const double two_pi = 6.283185307179586476925286766559;
        double ang = (double)pos * a.inv_freq[fi];
        ang -= two_pi * rint(ang * (1.0 / two_pi));
        a.rope[(size_t)m * (a.head_dim / 2) + fi] = float2{(float)cos(ang), (float)sin(ang)};
    }
    int tok;
    if (a.source == 0) tok = a.tokens[m];
    else if (j == 0) tok = a.anchor[b];
    else if (a.source == 1) tok = a.mask_id;
    else if (a.source == 3) tok = j < a.quad_k ? a.draft[b * (a.quad_k - 1) + j - 1] : a.mask_id;
    else tok = a.draft[b * (a.k_blk - 1) + j - 1];
    if (tok < 0 || tok >= a.vocab) {
        if (threadIdx.x == 0) atomicOr(a.status, DEV_BAD_TOKEN);
        tok = 0;
    }
    const uint16_t* e = a.embed + (size_t)tok * a.hidden;
    const size_t row = (size_t)m * a.hidden;
    const int chunks = a.hidden / 16;
    for (int c = threadIdx.x; c < chunks; c += blockDim.x) {   // 16 columns per thread
        float ss = 0.f;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int col = 16 * c + 8 * h;
            const uint4 w = *(const uint4*)(e + col);
            const uint4 gg = *(const uint4*)(a.gain + col);
            const uint32_t ew[4] = {w.x, w.y, w.z, w.w}, gw[4] = {gg.x, gg.y, gg.z, gg.w};
            float xv[8], xgv[8];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                xv[2 * q] = bf16_to_f32(ew[q] & 0xFFFFu);
                xv[2 * q + 1] = bf16_to_f32(ew[q] >> 16);
                xgv[2 * q] = xv[2 * q] * bf16_to_f32(gw[q] & 0xFFFFu);
                xgv[2 * q + 1] = xv[2 * q + 1] * bf16_to_f32(gw[q] >> 16);
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) ss += xv[q] * xv[q];
            *(float4*)(a.x + row + col) = float4{xv[0], xv[1], xv[2], xv[3]};
            *(float4*)(a.x + row + col + 4) = float4{xv[4], xv[5], xv[6], xv[7]};
            uint4 hi, lo;
            split8(xgv, hi, lo, a.plain & SITE_NORM);
            const size_t xi = split_index(m, col, a.hidden / 32);
            *(uint4*)(a.xg + xi) = hi;
            *(uint4*)(a.xg + xi + SPLIT_LO) = lo;
        }
        a.part_ss[(size_t)m * chunks + c] = ss;
    }
}

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
    launch(embed_kernel, dim3(a.M), dim3(256), s, a);
    return hipGetLastError();
}

// =====================================================================================
// Per-sequence finish: argmax of each block row (from the LM head's per-workgroup
// keys, or from given logits; lowest index among equal maxima), then draft
// extraction (d_j = argmax of draft row j), longest-prefix acceptance with the
// bonus token and the commit of L+1 rows, or a denoising step's commit: masked
// rows whose top-1 softmax probability exceeds the threshold take their argmax,
// else the most confident masked row does.  A refresh only commits k-1 rows.
// One workgroup per sequence, one wavefront per row.
// =====================================================================================
// the float value an argmax key was made from
__device__ __forceinline__ float argmax_key_value(unsigned long long key) {
    const uint32_t ord = (uint32_t)(key >> 32);
    return __uint_as_float((ord & 0x80000000u) ? (ord ^ 0x80000000u) : ~ord);
}

// Commit n more rows of sequence b.  Rows at or past max_len were never written (the QKV epilogue
// skipped them and set DEV_CAPACITY), so the length stops at max_len: every row below it is valid.
__device__ __forceinline__ void advance_length(const FinishArgs& a, int b, int n) {
    const int p = a.lengths[b] + n;
    if (p > a.max_len) {
        atomicOr(a.status, DEV_CAPACITY);
        a.lengths[b] = a.max_len;
    } else {
        a.lengths[b] = p;
    }
}

__global__ void __launch_bounds__(1024) finish_kernel(FinishArgs a) {
    __shared__ int32_t am[64];
    __shared__ float cf[64];
    const int b = blockIdx.x, k = a.k_blk;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const bool denoise = a.finish == FINISH_DENOISE;
    if (a.finish == FINISH_REFRESH) {
        if (threadIdx.x != 0) return;
        const int32_t* blk = a.block + (size_t)b * k;
        for (int j = 1; j < k; ++j)
            if (blk[j] == a.mask_id) atomicOr(a.status, DEV_MASK_LEFT);
        a.next_anchor[b] = blk[k - 1];
        advance_length(a, b, k - 1);
        return;
    }
    for (int jr = wave; jr < k; jr += nw) {
        const int m = b * k + jr;
        unsigned long long best = 0ull;
        float2 st = float2{-INFINITY, 0.f};   // softmax statistics (denoising only)
        if (a.part_keys) {
            const unsigned long long* pk = a.part_keys + (size_t)m * a.n_parts;
            int p = lane;
            for (; p + 192 < a.n_parts; p += 256)
                best = umax64(umax64(best, pk[p]), umax64(umax64(pk[p + 64], pk[p + 128]), pk[p + 192]));
            for (; p < a.n_parts; p += 64) best = umax64(best, pk[p]);
            if (denoise)
                for (int q = lane; q < a.n_parts; q += 64) st = lse_merge(st, a.part_lse[(size_t)m * a.n_parts + q]);
        } else {
            const float* lg = a.logits + (size_t)m * a.vocab;
            const int excl = denoise ? a.mask_id : -1;
            for (int n = lane; n < a.vocab; n += 64) {
                if (n == excl) continue;
                const float v = lg[n];
                best = umax64(best, argmax_key(v, (uint32_t)n));
                if (denoise) st = lse_merge(st, float2{v, 1.f});
            }
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) best = umax64(best, __shfl_xor(best, off));
        if (denoise) {
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) {
                const float2 o = float2{__shfl_xor(st.x, off), __shfl_xor(st.y, off)};
                st = lse_merge(st, o);
            }
        }
        if (lane == 0) {
            const int idx = argmax_key_index(best);
            am[jr] = idx;
            if (a.argmax_out) a.argmax_out[m] = idx;
            if (denoise) {
                // probability of the argmax token: exp(z_best - max) / sum (the max is z_best)
                const float c = expf(argmax_key_value(best) - st.x) / st.y;
                cf[jr] = c;
                if (a.conf_out) a.conf_out[m] = c;
            }
        }
    }
    __syncthreads();
    if (threadIdx.x != 0 || a.finish == FINISH_NONE) return;
    if (a.finish == FINISH_DRAFT) {
        for (int jj = 1; jj < k; ++jj) a.draft_out[(size_t)b * (k - 1) + jj - 1] = am[jj];
    } else if (denoise) {
        int32_t* blk = a.block + (size_t)b * k;
        int n_mask = 0, n_above = 0, top = -1;
        for (int j = 1; j < k; ++j) {
            if (blk[j] != a.mask_id) continue;
            ++n_mask;
            if (cf[j] > a.threshold) ++n_above;
            if (top < 0 || cf[j] > cf[top]) top = j;   // first of the most confident
        }
        for (int j = 1; j < k; ++j)
            if (blk[j] == a.mask_id && (n_above > 0 ? cf[j] > a.threshold : j == top)) blk[j] = am[j];
        const int n_commit = n_above > 0 ? n_above : (n_mask > 0 ? 1 : 0);
        a.n_committed[b] = n_commit;
        a.n_masked[b] = n_mask - n_commit;
    } else {
        const int32_t* dr = a.draft_in + (size_t)b * (k - 1);
        int L = 0;
        while (L < k - 1 && dr[L] == am[L]) ++L;
        a.accept_len[b] = L;
        for (int i = 0; i < k; ++i) a.committed[(size_t)b * k + i] = i < L ? dr[i] : (i == L ? am[L] : -1);
        a.next_anchor[b] = am[L];
        if (a.lengths) advance_length(a, b, L + 1);
    }
}

hipError_t launch_finish(const FinishArgs& a, hipStream_t s) {
    const int threads = a.finish == FINISH_REFRESH ? 64 : 64 * (a.k_blk < 16 ? a.k_blk : 16);
    launch(finish_kernel, dim3(a.batch), dim3(threads), s, a);
    return hipGetLastError();
}

// =====================================================================================
// Quadratic self-speculation (Sec. 3.4, Appendix C).  The block of each sequence is the
// chain [anchor, s_1 .. s_{qk-1}] followed by qk groups of qk masks (k_blk = qk(qk+1)
// rows).  The verifier token v_i of position P + i (i = 1..qk) comes from chain row i-1
// (AR), from mask 1 of group i-1 (diffusion), or from their mixture
// lambda * softmax(AR) + (1 - lambda) * softmax(diffusion).  Acceptance is Mode 3's; the
// next speculative tokens are the argmax of masks 2..qk of group L.
// =====================================================================================
// argmax of row m from the LM head's per-workgroup keys, in every lane of the wavefront
__device__ __forceinline__ int32_t row_argmax(const FinishArgs& a, int m, int lane) {
    const unsigned long long* pk = a.part_keys + (size_t)m * a.n_parts;
    unsigned long long best = 0ull;
    for (int p = lane; p < a.n_parts; p += 64) best = umax64(best, pk[p]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) best = umax64(best, __shfl_xor(best, off));
    return argmax_key_index(best);
}

// softmax statistics (max, sum of exp(z - max)) of row m, merged over the LM head's
// workgroups, in every lane of the wavefront
__device__ __forceinline__ float2 row_lse(const FinishArgs& a, int m, int lane) {
    float2 st = float2{-INFINITY, 0.f};
    for (int p = lane; p < a.n_parts; p += 64) st = lse_merge(st, a.part_lse[(size_t)m * a.n_parts + p]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) st = lse_merge(st, float2{__shfl_xor(st.x, off), __shfl_xor(st.y, off)});
    return st;
}

// Workgroup (sequence b and position i, vocabulary chunk ch): the argmax key over the chunk
// of lambda * exp(a_n - A) / SA + (1 - lambda) * exp(d_n - D) / SD (lowest index on ties),
// into ens_keys[(b * quad_k + i) * ens_chunks + ch].  Each thread has eight columns of both
// rows in flight at a time.
__global__ void __launch_bounds__(512) quad_ensemble_kernel(FinishArgs a) {
    __shared__ float2 st_s[2];
    __shared__ unsigned long long key_s[8];
    const int qk = a.quad_k, R = a.k_blk, V = a.vocab;
    const int bi = blockIdx.x, b = bi / qk, i = bi % qk, ch = blockIdx.y;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    if (wave < 2) {
        const float2 st = row_lse(a, b * R + (wave == 0 ? i : qk + i * qk), lane);
        if (lane == 0) st_s[wave] = st;
    }
    __syncthreads();
    const float2 sa = st_s[0], sd = st_s[1];
    const float ca = a.lambda / sa.y, cd = (1.0f - a.lambda) / sd.y;
    const float* la = a.ens_logits + ((size_t)b * 2 * qk + i) * V;
    const float* ld = a.ens_logits + ((size_t)b * 2 * qk + qk + i) * V;
    const int per = (V + a.ens_chunks - 1) / a.ens_chunks;
    const int n0 = ch * per, n1 = min(V, n0 + per), nt = blockDim.x;
    unsigned long long best = 0ull;
    for (int n = n0 + (int)threadIdx.x; n < n1; n += 8 * nt) {
        float xa[8], xd[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int j = n + u * nt;
            xa[u] = j < n1 ? la[j] : 0.f;
            xd[u] = j < n1 ? ld[j] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int j = n + u * nt;
            const float p = ca * expf(xa[u] - sa.x) + cd * expf(xd[u] - sd.x);
            if (j < n1) best = umax64(best, argmax_key(p, (uint32_t)j));
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) best = umax64(best, __shfl_xor(best, off));
    if (lane == 0) key_s[wave] = best;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long k2 = 0ull;
        for (int w = 0; w < nw; ++w) k2 = umax64(k2, key_s[w]);
        a.ens_keys[(size_t)bi * a.ens_chunks + ch] = k2;
    }
}

// One workgroup per sequence: verifier tokens, acceptance, commit, next anchor and the next
// speculative tokens.  draft_out may alias draft_in and next_anchor the anchor the pass read.
__global__ void __launch_bounds__(1024) quad_finish_kernel(FinishArgs a) {
    __shared__ int32_t v_s[64];
    __shared__ int L_s;
    const int b = blockIdx.x, qk = a.quad_k, R = a.k_blk;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    for (int i = wave; i < qk; i += nw) {
        int32_t v;
        if (a.lambda > 0.0f && a.lambda < 1.0f) {   // the ensemble kernel's per-chunk keys
            unsigned long long best = 0ull;
            for (int c = lane; c < a.ens_chunks; c += 64) best = umax64(best, a.ens_keys[(size_t)(b * qk + i) * a.ens_chunks + c]);
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) best = umax64(best, __shfl_xor(best, off));
            v = argmax_key_index(best);
        } else {
            v = row_argmax(a, b * R + (a.lambda >= 1.0f ? i : qk + i * qk), lane);
        }
        if (lane == 0) v_s[i] = v;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const int32_t* sp = a.draft_in + (size_t)b * (qk - 1);
        int L = 0;
        while (L < qk - 1 && sp[L] == v_s[L]) ++L;
        for (int i = 0; i < qk; ++i) a.committed[(size_t)b * qk + i] = i < L ? sp[i] : (i == L ? v_s[L] : -1);
        a.accept_len[b] = L;
        a.next_anchor[b] = v_s[L];
        if (a.lengths) advance_length(a, b, L + 1);
        L_s = L;
    }
    __syncthreads();
    const int L = L_s;
    for (int r = 2 + wave; r <= qk; r += nw) {
        const int32_t v = row_argmax(a, b * R + qk + L * qk + r - 1, lane);
        if (lane == 0) a.draft_out[(size_t)b * (qk - 1) + r - 2] = v;
    }
}

hipError_t launch_quad_ensemble(const FinishArgs& a, hipStream_t s) {
    launch(quad_ensemble_kernel, dim3(a.batch * a.quad_k, a.ens_chunks), dim3(512), s, a);
    return hipGetLastError();
}

hipError_t launch_quad_finish(const FinishArgs& a, hipStream_t s) {
    launch(quad_finish_kernel, dim3(a.batch), dim3(64 * (a.quad_k < 16 ? a.quad_k : 16)), s, a);
    return hipGetLastError();
}

// =====================================================================================
// Weight packing into MFMA B-operand tiles, and a fill kernel.
// =====================================================================================
__global__ void __launch_bounds__(256) pack_kernel(PackArgs p) {
    const size_t total = (size_t)p.n_tiles * p.ksteps * 64;
    for (size_t c = (size_t)blockIdx.x * blockDim.x + threadIdx.x; c < total; c += (size_t)gridDim.x * blockDim.x) {
        const int lane = (int)(c % 64);
        const size_t ts = c / 64;
        const int s = (int)(ts % p.ksteps);
        const int t = (int)(ts / p.ksteps);
        const int col = lane & 15;
        const int kk = 32 * s + 8 * (lane >> 4);
        const uint16_t* row = nullptr;
        if (p.kind == PACK_LINEAR) {
            const int n = 16 * t + col;
            if (n < p.out_dim) row = p.src0 + (size_t)n * p.in_dim;
        } else if (p.kind == PACK_QKV) {
            const int D = p.head_dim, tph = D / 16;
            const int hh = t / tph, u = t % tph;
            const int fi = 8 * u + (col & 7);
            const int n = hh * D + ((col < 8) ? fi : D / 2 + fi);
            if (n < p.rows0) row = p.src0 + (size_t)n * p.in_dim;
            else if (n < p.rows0 + p.rows1) row = p.src1 + (size_t)(n - p.rows0) * p.in_dim;
            else if (n < p.out_dim) row = p.src2 + (size_t)(n - p.rows0 - p.rows1) * p.in_dim;
        } else {
            const int f = 8 * t + (col & 7);
            if (f < p.rows0) row = ((col < 8) ? p.src0 : p.src1) + (size_t)f * p.in_dim;
        }
        uint4 v = {0u, 0u, 0u, 0u};
        if (row && kk < p.in_dim) v = *(const uint4*)(row + kk);
        p.dst[c] = v;
    }
}

hipError_t launch_pack(const PackArgs& a, hipStream_t s) {
    const size_t total = (size_t)a.n_tiles * a.ksteps * 64;
    size_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    launch(pack_kernel, dim3((unsigned)blocks), dim3(256), s, a);
    return hipGetLastError();
}

__global__ void fill_zero_kernel(uint32_t* p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = 0u;
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) {
    const size_t n = bytes / 4;
    size_t blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    if (blocks == 0) return hipSuccess;
    launch(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), s, (uint32_t*)p, n);
    return hipGetLastError();
}

__global__ void copy_u32_kernel(const uint32_t* src, uint32_t* dst) {
    if (threadIdx.x == 0) *dst = *src;
}

hipError_t launch_copy_u32(const uint32_t* src, uint32_t* dst, hipStream_t s) {
    launch(copy_u32_kernel, dim3(1), dim3(64), s, src, dst);
    return hipGetLastError();
}

}  // namespace nld

#ifdef NLD_TIMELINE
// copies the phase timestamps (8 x 8192 x 8 uint64) to host memory, or clears them (host == NULL)
extern "C" int nld_timeline_read(void* host, size_t bytes) {
    if (!host) {
        static unsigned long long zero[8 * 8192 * 8];
        return (int)hipMemcpyToSymbol(HIP_SYMBOL(nld::g_timeline), zero, sizeof(zero), 0, hipMemcpyHostToDevice);
    }
    return (int)hipMemcpyFromSymbol(host, HIP_SYMBOL(nld::g_timeline), bytes, 0, hipMemcpyDeviceToHost);
}
#endif
