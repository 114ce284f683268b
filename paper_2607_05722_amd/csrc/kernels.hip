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
// wavefront load).  No kernel communicates across workgroups: every output
// element is finished by exactly one workgroup (agent-scope fences and
// same-address atomics cost tens of microseconds per kernel on this chip).

#include "nld_internal.h"

#include <math.h>

namespace nld {

static constexpr uint32_t DEV_BAD_TOKEN = 0x1u;
static constexpr uint32_t DEV_CAPACITY = 0x2u;
static constexpr uint32_t DEV_BAD_LENGTH = 0x4u;

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
// GEMM epilogues.  v holds C[4g+i][r] of a 16x16 output tile (rows mbase..+16, packed
// column tile t); lane = 16g + r.  inv(i) is the RMSNorm scale of row mbase+4g+i.
// =====================================================================================
template <typename InvFn>
__device__ __forceinline__ void epi_qkv(const GemmArgs& a, f32x4_t v, int mbase, int t, int lane, InvFn inv) {
    const int r = lane & 15, g = lane >> 4;
    const int D = a.head_dim;
    const int tiles_per_head = D / 16;
    const int hh = t / tiles_per_head, u = t % tiles_per_head;
    const int fi = 8 * u + (r & 7);             // rotary frequency index, < D/2
    const int dim = (r < 8) ? fi : D / 2 + fi;  // lanes r and r^8 hold the pair (fi, fi + D/2)
    const int nq = a.n_q_heads, nkv = a.n_kv_heads;
    const int kind = hh < nq ? 0 : (hh < nq + nkv ? 1 : 2);
    const double inv_freq = exp2(-(2.0 * (double)fi / (double)D) * a.log2_base);
    const double two_pi = 6.283185307179586476925286766559;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = mbase + 4 * g + i;
        const bool ok = m < a.M;
        const int mm = ok ? m : 0;
        const float y = v[i] * inv(i);
        const float partner = __shfl_xor(y, 8);
        const int b = mm / a.k_blk, j = mm % a.k_blk;
        const int pos = committed_length(a.lengths, b, a.max_len, a.status) + j;
        float out = y;
        if (kind < 2) {
            double ang = (double)pos * inv_freq;
            ang -= two_pi * rint(ang / two_pi);
            float sn, cs;
            sincosf((float)ang, &sn, &cs);
            out = (r < 8) ? (y * cs - partner * sn) : (y * cs + partner * sn);
        }
        if (!ok) continue;
        const uint16_t ob = (uint16_t)f32_to_bf16(out);
        if (kind == 0) {
            a.q_out[(size_t)m * (nq * D) + hh * D + dim] = ob;
        } else if (pos >= a.max_len) {
            atomicOr(a.status, DEV_CAPACITY);
        } else if (kind == 1) {
            const int kvh = hh - nq;
            a.kc[((size_t)(b * nkv + kvh) * a.max_len + pos) * D + dim] = ob;
        } else {
            const int kvh = hh - nq - nkv;
            a.vc[(((size_t)(b * nkv + kvh) * (a.max_len / 64) + pos / 64) * D + dim) * 64 + (pos & 63)] = ob;
        }
    }
}

template <typename InvFn>
__device__ __forceinline__ void epi_swiglu(const GemmArgs& a, f32x4_t v, int mbase, int t, int lane, InvFn inv) {
    const int r = lane & 15, g = lane >> 4;
    const int col = 8 * t + (r & 7);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = mbase + 4 * g + i;
        const float y = v[i] * inv(i);
        const float partner = __shfl_xor(y, 8);   // lanes r < 8 hold gate columns, r^8 the matching up columns
        if (m < a.M && r < 8 && col < a.ffn) {
            const float gate = y, up = partner;
            const float act = gate / (1.0f + expf(-gate)) * up;
            a.act[(size_t)m * a.ffn + col] = (uint16_t)f32_to_bf16(act);
        }
    }
}

// Returns, in every lane with r == 0, the argmax keys of rows mbase+4g+i over this tile.
template <typename InvFn>
__device__ __forceinline__ void epi_lmhead(const GemmArgs& a, f32x4_t v, int mbase, int t, int lane, InvFn inv,
                                           unsigned long long (&key_run)[4]) {
    const int r = lane & 15, g = lane >> 4;
    const int n = t * 16 + r;
    const bool col_ok = n < a.vocab;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = mbase + 4 * g + i;
        const bool ok = m < a.M;
        const float y = v[i] * inv(i);
        if (ok && col_ok && a.logits) a.logits[(size_t)m * a.vocab + n] = y;
        unsigned long long key = (ok && col_ok) ? argmax_key(y, (uint32_t)n) : 0ull;
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) key = umax64(key, __shfl_xor(key, off));
        key_run[i] = umax64(key_run[i], key);
    }
}

__device__ __forceinline__ void epi_resid(const GemmArgs& a, f32x4_t v, int mbase, int t, int lane) {
    const int r = lane & 15, g = lane >> 4;
    const int N = a.n_tiles * 16;
    const int n = t * 16 + r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = mbase + 4 * g + i;
        if (m < a.M) a.x[(size_t)m * N + n] += v[i];
    }
}

// =====================================================================================
// Normed multi-tile GEMM (M <= 16 rows).  A workgroup of NW wavefronts owns a
// contiguous range of output tiles; wavefront w owns the reduction slice
// [32*KS*w, 32*KS*(w+1)).  At the start each wavefront loads its slice of the
// residual stream x, multiplies by the RMSNorm gain and keeps the bf16 operand in
// registers for all tiles; the per-row sum of squares is reduced across the
// wavefronts (fixed order) to the RMSNorm scale.  Weight tiles are streamed with
// one tile in flight ahead of the one being multiplied; per tile the NW partial
// products meet in LDS and one wavefront (rotating) runs the epilogue.
// =====================================================================================
template <int KS, int EPI>
__global__ void __launch_bounds__(512) gemm_norm_kernel(GemmArgs a) {
    __shared__ f32x4_t red[2][16][64];
    __shared__ float ss_part[16][16];
    __shared__ float inv_s[16];
    __shared__ unsigned long long key_s[16][16];

    const int NW = blockDim.x >> 6;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int T = a.n_tiles, G = gridDim.x;
    const int tb = (int)((long long)T * blockIdx.x / G);
    const int te = (int)((long long)T * (blockIdx.x + 1) / G);
    const int s0 = wave * KS;

    constexpr int KH = KS / 2;   // weights stream in half-tiles: one half-tile in flight ahead
    auto load_w = [&](int t, int half, uint4 (&buf)[KH]) {
        const uint4* p = a.W + ((size_t)t * a.ksteps + s0 + half * KH) * 64 + lane;
#pragma unroll
        for (int s = 0; s < KH; ++s) buf[s] = p[(size_t)s * 64];
    };
    uint4 wb0[KH], wb1[KH];
    if (tb < te) load_w(tb, 0, wb0);

    // operand slice: row r, columns 32*(s0+s) + 8g .. +8
    uint4 areg[KS];
    float ss = 0.f;
    const bool row_ok = r < a.M;
    const float* xr = a.x_in + (size_t)(row_ok ? r : 0) * a.K;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const int col = 32 * (s0 + s) + 8 * g;
        uint4 packed = {0u, 0u, 0u, 0u};
        if (row_ok) {
            const float4 x0 = *(const float4*)(xr + col);
            const float4 x1 = *(const float4*)(xr + col + 4);
            const uint4 gg = *(const uint4*)(a.gain + col);
            ss += x0.x * x0.x + x0.y * x0.y + x0.z * x0.z + x0.w * x0.w;
            ss += x1.x * x1.x + x1.y * x1.y + x1.z * x1.z + x1.w * x1.w;
            packed.x = f32_to_bf16(x0.x * bf16_to_f32(gg.x & 0xFFFFu)) | (f32_to_bf16(x0.y * bf16_to_f32(gg.x >> 16)) << 16);
            packed.y = f32_to_bf16(x0.z * bf16_to_f32(gg.y & 0xFFFFu)) | (f32_to_bf16(x0.w * bf16_to_f32(gg.y >> 16)) << 16);
            packed.z = f32_to_bf16(x1.x * bf16_to_f32(gg.z & 0xFFFFu)) | (f32_to_bf16(x1.y * bf16_to_f32(gg.z >> 16)) << 16);
            packed.w = f32_to_bf16(x1.z * bf16_to_f32(gg.w & 0xFFFFu)) | (f32_to_bf16(x1.w * bf16_to_f32(gg.w >> 16)) << 16);
        }
        areg[s] = packed;
    }
    ss += __shfl_xor(ss, 16);
    ss += __shfl_xor(ss, 32);
    if (g == 0) ss_part[wave][r] = ss;
    __syncthreads();
    if (threadIdx.x < 16) {
        float tot = 0.f;
        for (int w = 0; w < NW; ++w) tot += ss_part[w][threadIdx.x];
        inv_s[threadIdx.x] = ((int)threadIdx.x < a.M) ? 1.0f / sqrtf(tot / (float)a.K + a.eps) : 0.f;
    }
    __syncthreads();
    auto inv = [&](int i) { return inv_s[4 * g + i]; };

    unsigned long long key_run[4] = {0ull, 0ull, 0ull, 0ull};
    auto finish_tile = [&](int t, int parity) {
        f32x4_t v = red[parity][0][lane];
        for (int w = 1; w < NW; ++w) v += red[parity][w][lane];
        if constexpr (EPI == EPI_QKV) epi_qkv(a, v, 0, t, lane, inv);
        else if constexpr (EPI == EPI_SWIGLU) epi_swiglu(a, v, 0, t, lane, inv);
        else epi_lmhead(a, v, 0, t, lane, inv, key_run);
    };

    for (int t = tb; t < te; ++t) {
        load_w(t, 1, wb1);
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KH; ++s) acc = mfma_16x16x32(areg[s], wb0[s], acc);
        if (t + 1 < te) load_w(t + 1, 0, wb0);
#pragma unroll
        for (int s = 0; s < KH; ++s) acc = mfma_16x16x32(areg[KH + s], wb1[s], acc);
        const int parity = (t - tb) & 1;
        red[parity][wave][lane] = acc;
        __syncthreads();
        if (wave == (t - tb) % NW) finish_tile(t, parity);
    }

    if constexpr (EPI == EPI_LMHEAD) {
        // one argmax key per row for this workgroup
        if (r == 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i) key_s[wave][4 * g + i] = key_run[i];
        }
        __syncthreads();
        if ((int)threadIdx.x < a.M && threadIdx.x < 16) {
            unsigned long long best = 0ull;
            for (int w = 0; w < NW; ++w) best = umax64(best, key_s[w][threadIdx.x]);
            a.part_keys[(size_t)threadIdx.x * a.n_parts + blockIdx.x] = best;
        }
    }
}

bool gemm_norm_supported(int ks) { return ks == 4 || ks == 8 || ks == 16 || ks == 20; }  // even: half-tiles

template <int KS>
static hipError_t launch_norm_ks(int epi, int waves, int grid, const GemmArgs& a, hipStream_t s) {
    const dim3 blk(waves * 64);
    switch (epi) {
        case EPI_QKV: gemm_norm_kernel<KS, EPI_QKV><<<grid, blk, 0, s>>>(a); break;
        case EPI_SWIGLU: gemm_norm_kernel<KS, EPI_SWIGLU><<<grid, blk, 0, s>>>(a); break;
        case EPI_LMHEAD: gemm_norm_kernel<KS, EPI_LMHEAD><<<grid, blk, 0, s>>>(a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_gemm_norm(int epi, int ks, int waves, int grid, const GemmArgs& a, hipStream_t s) {
    if (waves < 1 || waves > 8) return hipErrorInvalidValue;
    switch (ks) {
        case 4: return launch_norm_ks<4>(epi, waves, grid, a, s);
        case 8: return launch_norm_ks<8>(epi, waves, grid, a, s);
        case 16: return launch_norm_ks<16>(epi, waves, grid, a, s);
        case 20: return launch_norm_ks<20>(epi, waves, grid, a, s);
        default: return hipErrorInvalidValue;
    }
}

// =====================================================================================
// Streamed GEMM: out[m][n] = sum_k A[m][k] W[n][k] for 16*MT rows x 16*CT columns per
// workgroup; the NW wavefronts split the reduction, each streaming its slice of the
// weights and of the bf16 activations with one batch in flight ahead of the MFMAs.
// Used for the O and down projections (residual epilogue) and, for M > 16, for
// every projection (the RMSNorm operand then comes from rmsnorm_prep_kernel).
// =====================================================================================
template <int MT, int CT>
struct Batch {
    static constexpr int U = (CT + MT <= 2) ? 8 : ((CT + MT <= 5) ? 4 : 2);
    uint4 w[U][CT];
    uint4 x[U][MT];
};

template <int MT, int CT, int NW, int EPI>
__global__ void __launch_bounds__(NW * 64) gemm_stream_kernel(GemmArgs a) {
    typedef Batch<MT, CT> B;
    constexpr int U = B::U;
    __shared__ f32x4_t red[NW][MT * CT][64];
    __shared__ unsigned long long key_s[16 * MT];

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
        const int m = m0 + mt * 16 + r;
        aok[mt] = m < a.M;
        ap[mt] = a.A + (size_t)(aok[mt] ? m : 0) * a.lda + 8 * g;
    }

    f32x4_t acc[MT][CT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[mt][ct] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const uint4 zero4 = {0u, 0u, 0u, 0u};
    auto load = [&](int s, B& buf) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int ss = s + u;
            const bool in = ss < s_end;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) buf.w[u][ct] = in ? wp[ct][(size_t)ss * 64] : zero4;
            const int kcol = ss * 32 + 8 * g;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                buf.x[u][mt] = (in && aok[mt] && kcol < a.K) ? *(const uint4*)(ap[mt] + (size_t)ss * 32) : zero4;
        }
    };
    auto compute = [&](const B& buf) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int ct = 0; ct < CT; ++ct) acc[mt][ct] = mfma_16x16x32(buf.x[u][mt], buf.w[u][ct], acc[mt][ct]);
    };

    B b0, b1;
    load(s_begin, b0);
    for (int s = s_begin; s < s_end; s += 2 * U) {
        load(s + U, b1);
        compute(b0);
        load(s + 2 * U, b0);
        compute(b1);
    }

#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) red[wave][mt * CT + ct][lane] = acc[mt][ct];
    if constexpr (EPI == EPI_LMHEAD) {
        if (threadIdx.x < 16 * MT) key_s[threadIdx.x] = 0ull;
    }
    __syncthreads();
    for (int ti = wave; ti < MT * CT; ti += NW) {
        f32x4_t v = red[0][ti][lane];
#pragma unroll
        for (int w = 1; w < NW; ++w) v += red[w][ti][lane];
        const int mt = ti / CT, ct = ti % CT;
        const int t = t0 + ct;
        if (t >= a.n_tiles) continue;
        const int mbase = m0 + 16 * mt;
        auto inv = [&](int i) {
            const int m = mbase + 4 * g + i;
            return m < a.M ? a.inv_rms[m] : 0.f;
        };
        if constexpr (EPI == EPI_RESID) epi_resid(a, v, mbase, t, lane);
        else if constexpr (EPI == EPI_QKV) epi_qkv(a, v, mbase, t, lane, inv);
        else if constexpr (EPI == EPI_SWIGLU) epi_swiglu(a, v, mbase, t, lane, inv);
        else {
            unsigned long long kr[4] = {0ull, 0ull, 0ull, 0ull};
            epi_lmhead(a, v, mbase, t, lane, inv, kr);
            if (r == 0) {
#pragma unroll
                for (int i = 0; i < 4; ++i) atomicMax(&key_s[16 * mt + 4 * g + i], kr[i]);
            }
        }
    }
    if constexpr (EPI == EPI_LMHEAD) {
        __syncthreads();
        if (threadIdx.x < 16 * MT) {
            const int m = m0 + threadIdx.x;
            if (m < a.M) a.part_keys[(size_t)m * a.n_parts + blockIdx.x] = key_s[threadIdx.x];
        }
    }
}

template <int EPI, int MT>
static hipError_t launch_stream_ct(int ct, int nw, dim3 grid, const GemmArgs& a, hipStream_t s) {
    if (ct == 1 && nw == 8) gemm_stream_kernel<MT, 1, 8, EPI><<<grid, 512, 0, s>>>(a);
    else if (ct == 2 && nw == 8) gemm_stream_kernel<MT, 2, 8, EPI><<<grid, 512, 0, s>>>(a);
    else if (ct == 4 && nw == 4) gemm_stream_kernel<MT, 4, 4, EPI><<<grid, 256, 0, s>>>(a);
    else if (ct == 1 && nw == 4) gemm_stream_kernel<MT, 1, 4, EPI><<<grid, 256, 0, s>>>(a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

template <int EPI>
static hipError_t launch_stream_mt(int mt, int ct, int nw, dim3 grid, const GemmArgs& a, hipStream_t s) {
    switch (mt) {
        case 1: return launch_stream_ct<EPI, 1>(ct, nw, grid, a, s);
        case 2: return launch_stream_ct<EPI, 2>(ct, nw, grid, a, s);
        case 4: return launch_stream_ct<EPI, 4>(ct, nw, grid, a, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gemm_stream(int epi, int mt, int ct, int nw, int grid_x, int grid_y, const GemmArgs& a,
                              hipStream_t s) {
    const dim3 grid(grid_x, grid_y);
    switch (epi) {
        case EPI_QKV: return launch_stream_mt<EPI_QKV>(mt, ct, nw, grid, a, s);
        case EPI_RESID: return launch_stream_mt<EPI_RESID>(mt, ct, nw, grid, a, s);
        case EPI_SWIGLU: return launch_stream_mt<EPI_SWIGLU>(mt, ct, nw, grid, a, s);
        case EPI_LMHEAD: return launch_stream_mt<EPI_LMHEAD>(mt, ct, nw, grid, a, s);
        default: return hipErrorInvalidValue;
    }
}

// RMSNorm operand for the streamed path: xg = bf16(x * gain), inv_rms = 1/rms(x).
__global__ void __launch_bounds__(256) rmsnorm_prep_kernel(PrepArgs a) {
    __shared__ float red[4];
    const int m = blockIdx.x;
    const float* x = a.x + (size_t)m * a.hidden;
    float ss = 0.f;
    for (int c = threadIdx.x; c < a.hidden; c += blockDim.x) {
        const float v = x[c];
        ss += v * v;
        a.xg[(size_t)m * a.hidden + c] = (uint16_t)f32_to_bf16(v * bf16_to_f32(a.gain[c]));
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    if (threadIdx.x == 0) a.inv_rms[m] = 1.0f / sqrtf(((red[0] + red[1]) + (red[2] + red[3])) / (float)a.hidden + a.eps);
}

hipError_t launch_prep(const PrepArgs& a, hipStream_t s) {
    rmsnorm_prep_kernel<<<a.M, 256, 0, s>>>(a);
    return hipGetLastError();
}

// =====================================================================================
// Block-masked GQA attention.  Workgroup = (key split, sequence x KV head, row slice);
// one compute wavefront per 16 query rows of the GQA group (rows = heads of the
// group x block rows).  Keys stream through LDS in stages of 64 (K rows and the
// cache's transposed V tile, XOR-swizzled for conflict-free operand reads), double
// buffered: the next stage's global loads are in flight while the current one is
// multiplied.  S^T = K Q^T on MFMA puts one query row per lane column, so a row's
// softmax statistics live in lanes r, r+16, r+32, r+48 and P^T is already the B
// operand of O^T = V^T P^T.  Online softmax in base 2, fp32.
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

template <int D>
__global__ void __launch_bounds__(512) attention_kernel(AttnArgs a) {
    typedef AttnCfg<D> C;
    constexpr int DC = D / 32;
    constexpr int DT = D / 16;
    constexpr int CPT_MAX = C::CHUNKS / 256;   // chunks per thread with >= 4 wavefronts
    __shared__ uint4 lds_k[2][C::KCHUNKS];
    __shared__ uint4 lds_v[2][C::VCHUNKS];

    const int nthreads = blockDim.x;
    const int cpt = C::CHUNKS / nthreads;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int split = blockIdx.x, unit = blockIdx.y;
    const int nkv = a.n_kv_heads, G = a.n_q_heads / nkv;
    const int b = unit / nkv, kvh = unit % nkv;
    const int k = a.k_blk, R = G * k;
    const int HD = a.n_q_heads * D;
    const int rt = blockIdx.z * 8 + wave;            // this wavefront's row tile
    const bool computes = wave < 8 && rt < a.row_tiles;
    const int row = rt * 16 + r;
    const bool row_ok = computes && row < R;
    const int hl = row_ok ? row / k : 0, j = row_ok ? row % k : 0;
    const int m = b * k + j;
    const int head = kvh * G + hl;

    int P = a.lengths[b];
    P = P < 0 ? 0 : (P > a.max_len ? a.max_len : P);
    const int T = min(P + k, a.max_len);
    const int kbeg = split * a.chunk;
    const int kend = min(kbeg + a.chunk, T);
    const bool bidir_row = (a.mode == 1) && (j >= a.bidir_from);

    const size_t head_off = (size_t)(b * nkv + kvh) * a.max_len * D;
    const uint16_t* kbase = a.kc + head_off;
    const uint16_t* vbase = a.vc + head_off;

    // stage loads: chunk q < KCHUNKS is K row q/KCH, chunk q%KCH; otherwise V row (q-KCHUNKS)/8, chunk %8
    uint4 stg[CPT_MAX];
    auto gload = [&](int kb) {
#pragma unroll
        for (int i = 0; i < CPT_MAX; ++i) {
            if (i >= cpt) break;
            const int q = threadIdx.x + i * nthreads;
            if (q < C::KCHUNKS) {
                stg[i] = *(const uint4*)(kbase + (size_t)kb * D + (size_t)q * 8);
            } else {
                const int qv = q - C::KCHUNKS;
                stg[i] = *(const uint4*)(vbase + (size_t)(kb >> 6) * D * 64 + (size_t)qv * 8);
                const int key0 = kb + 8 * (qv & 7);
                if (key0 + 8 > kend) {      // zero V beyond the valid keys (cache rows there may hold anything)
                    uint32_t w[4] = {stg[i].x, stg[i].y, stg[i].z, stg[i].w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const bool lo = key0 + 2 * e < kend, hi = key0 + 2 * e + 1 < kend;
                        w[e] = (lo ? (w[e] & 0xFFFFu) : 0u) | (hi ? (w[e] & 0xFFFF0000u) : 0u);
                    }
                    stg[i] = uint4{w[0], w[1], w[2], w[3]};
                }
            }
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < CPT_MAX; ++i) {
            if (i >= cpt) break;
            const int q = threadIdx.x + i * nthreads;
            if (q < C::KCHUNKS) {
                const int kr = q / C::KCH, c = q % C::KCH;
                lds_k[buf][kr * C::KCH + (c ^ kswz<D>(kr))] = stg[i];
            } else {
                const int qv = q - C::KCHUNKS;
                const int d = qv >> 3, c = qv & 7;
                lds_v[buf][d * 8 + (c ^ vswz(d))] = stg[i];
            }
        }
    };

    const uint4 zero4 = {0u, 0u, 0u, 0u};
    uint4 qb[DC];
#pragma unroll
    for (int c = 0; c < DC; ++c)
        qb[c] = row_ok ? *(const uint4*)(a.q + (size_t)m * HD + head * D + 32 * c + 8 * g) : zero4;

    f32x4_t acc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_part = 0.f;

    const int nstages = kend > kbeg ? (kend - kbeg + 63) / 64 : 0;
    if (nstages > 0) {
        gload(kbeg);
        lstore(0);
    }
    __syncthreads();
    for (int st = 0; st < nstages; ++st) {
        const int kb = kbeg + 64 * st;
        const int buf = st & 1;
        if (st + 1 < nstages) gload(kb + 64);
        if (computes) {
            f32x4_t s[4];
#pragma unroll
            for (int tau = 0; tau < 4; ++tau) {
                const int kr = stage_key(tau, r);
                s[tau] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int c = 0; c < DC; ++c) {
                    const uint4 kv4 = lds_k[buf][kr * C::KCH + ((4 * c + g) ^ kswz<D>(kr))];
                    s[tau] = mfma_16x16x32(kv4, qb[c], s[tau]);
                }
            }
            float sv[16];
            float mloc = -INFINITY;
#pragma unroll
            for (int tau = 0; tau < 4; ++tau)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int key = kb + stage_key(tau, 4 * g + i);
                    const bool vis = key < kend && (key < P || (key - P) <= j || bidir_row);
                    const float x = vis ? s[tau][i] * a.scale_log2 : -INFINITY;
                    sv[tau * 4 + i] = x;
                    mloc = fmaxf(mloc, x);
                }
            mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
            mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
            const float m_new = fmaxf(m_run, mloc);
            float alpha = 1.f;
            float p[16];
            if (m_new == -INFINITY) {
#pragma unroll
                for (int e = 0; e < 16; ++e) p[e] = 0.f;
            } else {
                alpha = exp2f(m_run - m_new);
#pragma unroll
                for (int e = 0; e < 16; ++e) p[e] = exp2f(sv[e] - m_new);
            }
            float psum = 0.f;
#pragma unroll
            for (int e = 0; e < 16; ++e) psum += p[e];
            l_part = l_part * alpha + psum;
            m_run = m_new;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) acc[dt] *= alpha;
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                // slot jj of lane group g <-> key kb + 32ks + 8g + jj
                uint4 pop;
                const float* pp = p + 8 * ks;
                pop.x = f32_to_bf16(pp[0]) | (f32_to_bf16(pp[1]) << 16);
                pop.y = f32_to_bf16(pp[2]) | (f32_to_bf16(pp[3]) << 16);
                pop.z = f32_to_bf16(pp[4]) | (f32_to_bf16(pp[5]) << 16);
                pop.w = f32_to_bf16(pp[6]) | (f32_to_bf16(pp[7]) << 16);
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
                    const int d = 16 * dt + r;
                    const uint4 vop = lds_v[buf][d * 8 + ((4 * ks + g) ^ vswz(d))];
                    acc[dt] = mfma_16x16x32(vop, pop, acc[dt]);
                }
            }
        }
        if (st + 1 < nstages) lstore(buf ^ 1);
        __syncthreads();
    }

    if (!computes) return;
    float l_tot = l_part + __shfl_xor(l_part, 16);
    l_tot += __shfl_xor(l_tot, 32);

    if (a.n_splits == 1) {
        if (row_ok) {
            const float inv = 1.0f / l_tot;
            uint16_t* op = a.o + (size_t)m * HD + head * D;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int i = 0; i < 4; ++i) op[16 * dt + 4 * g + i] = (uint16_t)f32_to_bf16(acc[dt][i] * inv);
        }
        return;
    }
    const size_t pbase = ((size_t)unit * a.n_splits + split) * a.rows_pad + row;
    float* po = a.part_o + pbase * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) *(float4*)(po + 16 * dt + 4 * g) = float4{acc[dt][0], acc[dt][1], acc[dt][2], acc[dt][3]};
    if (g == 0) *(float2*)(a.part_ml + pbase * 2) = float2{m_run, l_tot};
}

// Merge of the key splits: one workgroup per (unit, query row), one thread per head dim.
template <int D>
__global__ void __launch_bounds__(D) attention_combine_kernel(AttnArgs a) {
    const int unit = blockIdx.x, rw = blockIdx.y, d = threadIdx.x;
    const int nkv = a.n_kv_heads, G = a.n_q_heads / nkv;
    const int b = unit / nkv, kvh = unit % nkv, k = a.k_blk;
    const size_t ubase = (size_t)unit * a.n_splits * a.rows_pad + rw;
    float mx = -INFINITY;
    for (int sp = 0; sp < a.n_splits; ++sp) mx = fmaxf(mx, a.part_ml[(ubase + (size_t)sp * a.rows_pad) * 2]);
    float num = 0.f, den = 0.f;
    int sp = 0;
    for (; sp + 4 <= a.n_splits; sp += 4) {
        float ms[4], ls[4], os[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const size_t pb = ubase + (size_t)(sp + e) * a.rows_pad;
            ms[e] = a.part_ml[pb * 2];
            ls[e] = a.part_ml[pb * 2 + 1];
            os[e] = a.part_o[pb * D + d];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float w = (ms[e] == -INFINITY) ? 0.f : exp2f(ms[e] - mx);
            num += w * os[e];
            den += w * ls[e];
        }
    }
    for (; sp < a.n_splits; ++sp) {
        const size_t pb = ubase + (size_t)sp * a.rows_pad;
        const float ms = a.part_ml[pb * 2];
        const float w = (ms == -INFINITY) ? 0.f : exp2f(ms - mx);
        num += w * a.part_o[pb * D + d];
        den += w * a.part_ml[pb * 2 + 1];
    }
    const int hl = rw / k, j = rw % k;
    a.o[(size_t)(b * k + j) * a.n_q_heads * D + (kvh * G + hl) * D + d] = (uint16_t)f32_to_bf16(num / den);
}

hipError_t launch_attention(int head_dim, int waves, int zslices, int units, const AttnArgs& a, hipStream_t s) {
    const dim3 grid(a.n_splits, units, zslices);
    if (head_dim == 128) attention_kernel<128><<<grid, waves * 64, 0, s>>>(a);
    else if (head_dim == 64) attention_kernel<64><<<grid, waves * 64, 0, s>>>(a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_attention_combine(int head_dim, int units, int rows, const AttnArgs& a, hipStream_t s) {
    const dim3 grid(units, rows);
    if (head_dim == 128) attention_combine_kernel<128><<<grid, 128, 0, s>>>(a);
    else if (head_dim == 64) attention_combine_kernel<64><<<grid, 64, 0, s>>>(a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

// =====================================================================================
// Embedding gather of the block (block assembly per call kind) into the fp32 residual.
// =====================================================================================
__global__ void __launch_bounds__(256) embed_kernel(EmbedArgs a) {
    const int m = blockIdx.x;
    const int b = m / a.k_blk, j = m % a.k_blk;
    int tok;
    if (a.source == 0) tok = a.tokens[m];
    else if (j == 0) tok = a.anchor[b];
    else if (a.source == 1) tok = a.mask_id;
    else tok = a.draft[b * (a.k_blk - 1) + j - 1];
    if (tok < 0 || tok >= a.vocab) {
        if (threadIdx.x == 0) atomicOr(a.status, DEV_BAD_TOKEN);
        tok = 0;
    }
    const uint16_t* e = a.embed + (size_t)tok * a.hidden;
    for (int c = threadIdx.x; c < a.hidden; c += blockDim.x) a.x[(size_t)m * a.hidden + c] = bf16_to_f32(e[c]);
}

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
    embed_kernel<<<a.M, 256, 0, s>>>(a);
    return hipGetLastError();
}

// =====================================================================================
// Per-sequence finish: argmax of each block row (from the LM head's per-workgroup
// keys, or from given logits; lowest index among equal maxima), then draft
// extraction (d_j = argmax of draft row j) or longest-prefix acceptance with the
// bonus token and the commit of L+1 rows.  One workgroup per sequence, one
// wavefront per row.
// =====================================================================================
__global__ void __launch_bounds__(1024) finish_kernel(FinishArgs a) {
    __shared__ int32_t am[64];
    const int b = blockIdx.x, k = a.k_blk;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    for (int jr = wave; jr < k; jr += nw) {
        const int m = b * k + jr;
        unsigned long long best = 0ull;
        if (a.part_keys) {
            const unsigned long long* pk = a.part_keys + (size_t)m * a.n_parts;
            int p = lane;
            for (; p + 192 < a.n_parts; p += 256)
                best = umax64(umax64(best, pk[p]), umax64(umax64(pk[p + 64], pk[p + 128]), pk[p + 192]));
            for (; p < a.n_parts; p += 64) best = umax64(best, pk[p]);
        } else {
            const float* lg = a.logits + (size_t)m * a.vocab;
            for (int n = lane; n < a.vocab; n += 64) best = umax64(best, argmax_key(lg[n], (uint32_t)n));
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) best = umax64(best, __shfl_xor(best, off));
        if (lane == 0) {
            const int idx = argmax_key_index(best);
            am[jr] = idx;
            if (a.argmax_out) a.argmax_out[m] = idx;
        }
    }
    __syncthreads();
    if (threadIdx.x != 0 || a.finish == FINISH_NONE) return;
    if (a.finish == FINISH_DRAFT) {
        for (int jj = 1; jj < k; ++jj) a.draft_out[(size_t)b * (k - 1) + jj - 1] = am[jj];
    } else {
        const int32_t* dr = a.draft_in + (size_t)b * (k - 1);
        int L = 0;
        while (L < k - 1 && dr[L] == am[L]) ++L;
        a.accept_len[b] = L;
        for (int i = 0; i < k; ++i) a.committed[(size_t)b * k + i] = i < L ? dr[i] : (i == L ? am[L] : -1);
        a.next_anchor[b] = am[L];
        if (a.lengths) a.lengths[b] += L + 1;
    }
}

hipError_t launch_finish(const FinishArgs& a, hipStream_t s) {
    const int threads = 64 * (a.k_blk < 16 ? a.k_blk : 16);
    finish_kernel<<<a.batch, threads, 0, s>>>(a);
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
    pack_kernel<<<(unsigned)blocks, 256, 0, s>>>(a);
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
    fill_zero_kernel<<<(unsigned)blocks, 256, 0, s>>>((uint32_t*)p, n);
    return hipGetLastError();
}

}  // namespace nld
