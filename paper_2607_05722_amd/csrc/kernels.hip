// HIP kernels of the block-decode step for gfx950 (CDNA4).
//
// One forward pass over a k-token block per sequence (arXiv 2607.05722,
// Sec. 3.3, linear self-speculation) is:
//   embed -> L x [QKV GEMM (+RMSNorm scale, RoPE, K/V cache write),
//                 block-masked GQA attention (split over keys),
//                 O GEMM (+residual, next RMSNorm statistics),
//                 gate/up GEMM (+RMSNorm scale, SwiGLU),
//                 down GEMM (+residual, next RMSNorm statistics)]
//         -> LM-head GEMM (+final RMSNorm scale, per-tile argmax keys)
//         -> per-row argmax reduction + draft extraction / acceptance.
//
// The GEMMs are skinny (M = batch*k rows, usually 8..64): they are bound by
// streaming the bf16 weights from HBM.  Weights are pre-packed so that one
// 16-byte load per lane of a wavefront is exactly one MFMA B operand (1 KiB
// contiguous per wavefront load); activations are the A operand and come
// from L2.  A workgroup owns CT output tiles of 16 columns over the whole
// reduction; its NW wavefronts split the reduction and meet in LDS, so every
// output element is finished by exactly one workgroup and the epilogue runs
// in registers.

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

// =====================================================================================
// GEMM epilogues.  v holds C[4g+i][r] of the 16x16 output tile (rows mbase..+16,
// packed column tile t); lane = 16g + r.
// =====================================================================================
__device__ __forceinline__ void epi_resid(const GemmArgs& a, f32x4_t v, int mbase, int t, int lane) {
    const int r = lane & 15, g = lane >> 4;
    const int N = a.n_tiles * 16;
    const int n = t * 16 + r;
    const float gn = bf16_to_f32(a.gain[n]);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = mbase + 4 * g + i;
        float xn = 0.f;
        if (m < a.M) {
            float* xp = a.x + (size_t)m * N + n;
            xn = *xp + v[i];
            *xp = xn;
            a.xg[(size_t)m * N + n] = (uint16_t)f32_to_bf16(xn * gn);
        }
        float sq = xn * xn;
        sq += __shfl_xor(sq, 1);
        sq += __shfl_xor(sq, 2);
        sq += __shfl_xor(sq, 4);
        sq += __shfl_xor(sq, 8);
        if (r == 0 && m < a.M) a.part_ss[(size_t)m * a.n_tiles + t] = sq;
    }
}

__device__ __forceinline__ void epi_qkv(const GemmArgs& a, f32x4_t v, int mbase, int t, int lane) {
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
        const float y = v[i] * a.inv_rms[mm];
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

__device__ __forceinline__ void epi_swiglu(const GemmArgs& a, f32x4_t v, int mbase, int t, int lane) {
    const int r = lane & 15, g = lane >> 4;
    const int col = 8 * t + (r & 7);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = mbase + 4 * g + i;
        const bool ok = m < a.M;
        const float y = v[i] * a.inv_rms[ok ? m : 0];
        const float partner = __shfl_xor(y, 8);
        if (ok && r < 8 && col < a.ffn) {
            const float gate = y, up = partner;
            const float act = gate / (1.0f + expf(-gate)) * up;
            a.act[(size_t)m * a.ffn + col] = (uint16_t)f32_to_bf16(act);
        }
    }
}

__device__ __forceinline__ void epi_lmhead(const GemmArgs& a, f32x4_t v, int mbase, int t, int lane) {
    const int r = lane & 15, g = lane >> 4;
    const int n = t * 16 + r;
    const bool col_ok = n < a.vocab;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = mbase + 4 * g + i;
        const bool ok = m < a.M;
        const float y = v[i] * a.inv_rms[ok ? m : 0];
        if (ok && col_ok && a.logits) a.logits[(size_t)m * a.vocab + n] = y;
        unsigned long long key = (ok && col_ok) ? argmax_key(y, (uint32_t)n) : 0ull;
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) {
            const unsigned long long o = __shfl_xor(key, off);
            key = o > key ? o : key;
        }
        if (r == 0 && ok) a.part_keys[(size_t)m * a.n_tiles + t] = key;
    }
}

// =====================================================================================
// Skinny GEMM: out[m][n] = sum_k A[m][k] W[n][k] for 16*MT rows x 16*CT columns per
// workgroup, full reduction per workgroup split over NW wavefronts.
// =====================================================================================
template <int MT, int CT>
struct Batch {
    static constexpr int U = (CT + MT <= 2) ? 8 : ((CT + MT <= 5) ? 4 : 2);
    uint4 w[U][CT];
    uint4 x[U][MT];
};

template <int MT, int CT, int NW, int EPI>
__global__ void __launch_bounds__(NW * 64) gemm_skinny_kernel(GemmArgs a) {
    typedef Batch<MT, CT> B;
    constexpr int U = B::U;
    __shared__ f32x4_t red[NW][MT * CT][64];
    __shared__ int s_last;

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

    // reduce the NW partial tiles in LDS (fixed order), then run the epilogue
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) red[wave][mt * CT + ct][lane] = acc[mt][ct];
    __syncthreads();
    for (int ti = wave; ti < MT * CT; ti += NW) {
        f32x4_t v = red[0][ti][lane];
#pragma unroll
        for (int w = 1; w < NW; ++w) v += red[w][ti][lane];
        const int mt = ti / CT, ct = ti % CT;
        const int t = t0 + ct;
        if (t >= a.n_tiles) continue;
        const int mbase = m0 + 16 * mt;
        if constexpr (EPI == EPI_RESID) epi_resid(a, v, mbase, t, lane);
        else if constexpr (EPI == EPI_QKV) epi_qkv(a, v, mbase, t, lane);
        else if constexpr (EPI == EPI_SWIGLU) epi_swiglu(a, v, mbase, t, lane);
        else epi_lmhead(a, v, mbase, t, lane);
    }

    if constexpr (EPI == EPI_RESID) {
        // The last workgroup of this row group turns the per-tile sums of squares
        // into the next RMSNorm's per-row scale (fixed summation order).
        __threadfence();
        __syncthreads();
        if (threadIdx.x == 0) {
            const unsigned prev = atomicAdd(&a.counters[blockIdx.y], 1u);
            s_last = (prev == gridDim.x - 1) ? 1 : 0;
        }
        __syncthreads();
        if (s_last) {
            __threadfence();
            const int N = a.n_tiles * 16;
            for (int rr = wave; rr < 16 * MT; rr += NW) {
                const int m = m0 + rr;
                if (m >= a.M) break;
                float s = 0.f;
                for (int t = lane; t < a.n_tiles; t += 64) s += a.part_ss[(size_t)m * a.n_tiles + t];
                s = wave_sum(s);
                if (lane == 0) a.inv_rms_out[m] = 1.0f / sqrtf(s / (float)N + a.eps);
            }
            if (threadIdx.x == 0) __hip_atomic_store(&a.counters[blockIdx.y], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

template <int EPI, int MT>
static hipError_t launch_gemm_ct(int ct, int nw, dim3 grid, const GemmArgs& a, hipStream_t s) {
    if (ct == 1 && nw == 8) gemm_skinny_kernel<MT, 1, 8, EPI><<<grid, 512, 0, s>>>(a);
    else if (ct == 2 && nw == 8) gemm_skinny_kernel<MT, 2, 8, EPI><<<grid, 512, 0, s>>>(a);
    else if (ct == 4 && nw == 4) gemm_skinny_kernel<MT, 4, 4, EPI><<<grid, 256, 0, s>>>(a);
    else if (ct == 1 && nw == 4) gemm_skinny_kernel<MT, 1, 4, EPI><<<grid, 256, 0, s>>>(a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

template <int EPI>
static hipError_t launch_gemm_mt(int mt, int ct, int nw, dim3 grid, const GemmArgs& a, hipStream_t s) {
    switch (mt) {
        case 1: return launch_gemm_ct<EPI, 1>(ct, nw, grid, a, s);
        case 2: return launch_gemm_ct<EPI, 2>(ct, nw, grid, a, s);
        case 4: return launch_gemm_ct<EPI, 4>(ct, nw, grid, a, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gemm(int epi, int mt, int ct, int nw, int grid_x, int grid_y, const GemmArgs& a, hipStream_t s) {
    const dim3 grid(grid_x, grid_y);
    switch (epi) {
        case EPI_QKV: return launch_gemm_mt<EPI_QKV>(mt, ct, nw, grid, a, s);
        case EPI_RESID: return launch_gemm_mt<EPI_RESID>(mt, ct, nw, grid, a, s);
        case EPI_SWIGLU: return launch_gemm_mt<EPI_SWIGLU>(mt, ct, nw, grid, a, s);
        case EPI_LMHEAD: return launch_gemm_mt<EPI_LMHEAD>(mt, ct, nw, grid, a, s);
        default: return hipErrorInvalidValue;
    }
}

// =====================================================================================
// Block-masked GQA attention.  Workgroup = (key split, sequence x KV head); one
// wavefront per 16 query rows of the GQA group (rows = heads of the group x block
// rows).  S^T = K Q^T on MFMA puts one query row per lane column, so the softmax
// statistics of a row live in the four lanes r, r+16, r+32, r+48 and P^T is
// already the B operand of O^T = V^T P^T.  Online softmax in base 2 (fp32);
// splits are merged by the last workgroup of each unit.
// =====================================================================================
__device__ __forceinline__ uint32_t mask_pair(uint32_t w, bool lo_ok, bool hi_ok) {
    return (lo_ok ? (w & 0xFFFFu) : 0u) | (hi_ok ? (w & 0xFFFF0000u) : 0u);
}

template <int D>
__global__ void __launch_bounds__(1024) attention_kernel(AttnArgs a) {
    constexpr int DC = D / 32;
    constexpr int DT = D / 16;
    __shared__ int s_last;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int split = blockIdx.x, unit = blockIdx.y;
    const int nkv = a.n_kv_heads, G = a.n_q_heads / nkv;
    const int b = unit / nkv, kvh = unit % nkv;
    const int k = a.k_blk, R = G * k;
    const int HD = a.n_q_heads * D;
    const int row = wave * 16 + r;
    const bool row_ok = row < R;
    const int hl = row_ok ? row / k : 0, j = row_ok ? row % k : 0;
    const int m = b * k + j;
    const int head = kvh * G + hl;

    int P = a.lengths[b];
    P = P < 0 ? 0 : (P > a.max_len ? a.max_len : P);
    const int T = min(P + k, a.max_len);
    const int kbeg = split * a.chunk;
    const int kend = min(kbeg + a.chunk, T);
    const bool bidir_row = (a.mode == 1) && (j >= a.bidir_from);

    const uint4 zero4 = {0u, 0u, 0u, 0u};
    uint4 qb[DC];
#pragma unroll
    for (int c = 0; c < DC; ++c)
        qb[c] = row_ok ? *(const uint4*)(a.q + (size_t)m * HD + head * D + 32 * c + 8 * g) : zero4;

    const size_t head_off = (size_t)(b * nkv + kvh) * a.max_len * D;
    const uint16_t* kbase = a.kc + head_off;
    const uint16_t* vbase = a.vc + head_off;

    f32x4_t acc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_part = 0.f;

    for (int kb = kbeg; kb < kend; kb += 32) {
        f32x4_t s[2];
#pragma unroll
        for (int tau = 0; tau < 2; ++tau) {
            const int key = kb + 16 * tau + r;
            const bool kok = key < kend;
            const uint16_t* kp = kbase + (size_t)(kok ? key : 0) * D + 8 * g;
            s[tau] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < DC; ++c) {
                const uint4 kv4 = kok ? *(const uint4*)(kp + 32 * c) : zero4;
                s[tau] = mfma_16x16x32(kv4, qb[c], s[tau]);
            }
        }
        float sv[8];
        float mloc = -INFINITY;
#pragma unroll
        for (int tau = 0; tau < 2; ++tau)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key = kb + 16 * tau + 4 * g + i;
                const bool vis = key < kend && (key < P || (key - P) <= j || bidir_row);
                const float x = vis ? s[tau][i] * a.scale_log2 : -INFINITY;
                sv[tau * 4 + i] = x;
                mloc = fmaxf(mloc, x);
            }
        mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
        const float m_new = fmaxf(m_run, mloc);
        float alpha = 1.f;
        float p[8];
        if (m_new == -INFINITY) {
#pragma unroll
            for (int e = 0; e < 8; ++e) p[e] = 0.f;
        } else {
            alpha = exp2f(m_run - m_new);
#pragma unroll
            for (int e = 0; e < 8; ++e) p[e] = exp2f(sv[e] - m_new);
        }
        float psum = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) psum += p[e];
        l_part = l_part * alpha + psum;
        m_run = m_new;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) acc[dt] *= alpha;

        uint4 pop;
        pop.x = f32_to_bf16(p[0]) | (f32_to_bf16(p[1]) << 16);
        pop.y = f32_to_bf16(p[2]) | (f32_to_bf16(p[3]) << 16);
        pop.z = f32_to_bf16(p[4]) | (f32_to_bf16(p[5]) << 16);
        pop.w = f32_to_bf16(p[6]) | (f32_to_bf16(p[7]) << 16);

        const int tile = kb >> 6, off = kb & 63;
        const int k0 = kb + 4 * g, k1 = kb + 16 + 4 * g;
        const bool z0 = k0 + 3 < kend, z1 = k1 + 3 < kend;  // whole quads in range
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const int d = 16 * dt + r;
            const uint16_t* vp = vbase + ((size_t)tile * D + d) * 64 + off + 4 * g;
            uint2 lo = *(const uint2*)vp;
            uint2 hi = *(const uint2*)(vp + 16);
            if (!z0) {
                lo.x = mask_pair(lo.x, k0 < kend, k0 + 1 < kend);
                lo.y = mask_pair(lo.y, k0 + 2 < kend, k0 + 3 < kend);
            }
            if (!z1) {
                hi.x = mask_pair(hi.x, k1 < kend, k1 + 1 < kend);
                hi.y = mask_pair(hi.y, k1 + 2 < kend, k1 + 3 < kend);
            }
            const uint4 vop = {lo.x, lo.y, hi.x, hi.y};
            acc[dt] = mfma_16x16x32(vop, pop, acc[dt]);
        }
    }

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
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) po[16 * dt + 4 * g + i] = acc[dt][i];
    if (g == 0) {
        a.part_ml[pbase * 2] = m_run;
        a.part_ml[pbase * 2 + 1] = l_tot;
    }
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        const unsigned prev = atomicAdd(&a.counters[unit], 1u);
        s_last = (prev == (unsigned)a.n_splits - 1) ? 1 : 0;
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    const size_t ubase = (size_t)unit * a.n_splits * a.rows_pad;
    for (int idx = threadIdx.x; idx < R * D; idx += blockDim.x) {
        const int rw = idx / D, d = idx % D;
        float mx = -INFINITY;
        for (int sp = 0; sp < a.n_splits; ++sp) mx = fmaxf(mx, a.part_ml[(ubase + (size_t)sp * a.rows_pad + rw) * 2]);
        float num = 0.f, den = 0.f;
        for (int sp = 0; sp < a.n_splits; ++sp) {
            const size_t pb = ubase + (size_t)sp * a.rows_pad + rw;
            const float ms = a.part_ml[pb * 2];
            const float w = (ms == -INFINITY) ? 0.f : exp2f(ms - mx);
            num += w * a.part_o[pb * D + d];
            den += w * a.part_ml[pb * 2 + 1];
        }
        const int hl2 = rw / k, j2 = rw % k;
        a.o[(size_t)(b * k + j2) * HD + (kvh * G + hl2) * D + d] = (uint16_t)f32_to_bf16(num / den);
    }
    if (threadIdx.x == 0) __hip_atomic_store(&a.counters[unit], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

hipError_t launch_attention(int head_dim, int waves, int units, const AttnArgs& a, hipStream_t s) {
    const dim3 grid(a.n_splits, units);
    if (head_dim == 128) attention_kernel<128><<<grid, waves * 64, 0, s>>>(a);
    else if (head_dim == 64) attention_kernel<64><<<grid, waves * 64, 0, s>>>(a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

// =====================================================================================
// Embedding gather of the block (block assembly per call kind) + first RMSNorm stats.
// =====================================================================================
__global__ void __launch_bounds__(256) embed_kernel(EmbedArgs a) {
    __shared__ float red[4];
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
    float ss = 0.f;
    for (int c = threadIdx.x; c < a.hidden; c += blockDim.x) {
        const float v = bf16_to_f32(e[c]);
        a.x[(size_t)m * a.hidden + c] = v;
        a.xg[(size_t)m * a.hidden + c] = (uint16_t)f32_to_bf16(v * bf16_to_f32(a.gain[c]));
        ss += v * v;
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    if (threadIdx.x == 0) {
        const float tot = (red[0] + red[1]) + (red[2] + red[3]);
        a.inv_rms[m] = 1.0f / sqrtf(tot / (float)a.hidden + a.eps);
    }
}

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
    embed_kernel<<<a.M, 256, 0, s>>>(a);
    return hipGetLastError();
}

// =====================================================================================
// Per-row argmax (from LM-head tile keys, or from given logits) and the per-sequence
// finish: draft extraction (d_j = argmax of draft row j) or longest-prefix acceptance
// with the bonus token and the commit of L+1 rows.
// =====================================================================================
__global__ void __launch_bounds__(256) argmax_finish_kernel(ArgmaxArgs a) {
    __shared__ unsigned long long red[4];
    __shared__ int s_last;
    const int m = blockIdx.x;
    unsigned long long best = 0ull;
    if (a.part_keys) {
        const unsigned long long* pk = a.part_keys + (size_t)m * a.n_tiles;
        for (int t = threadIdx.x; t < a.n_tiles; t += blockDim.x) best = pk[t] > best ? pk[t] : best;
    } else {
        const float* lg = a.logits + (size_t)m * a.vocab;
        for (int n = threadIdx.x; n < a.vocab; n += blockDim.x) {
            const unsigned long long kk = argmax_key(lg[n], (uint32_t)n);
            best = kk > best ? kk : best;
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const unsigned long long o = __shfl_xor(best, off);
        best = o > best ? o : best;
    }
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = best;
    __syncthreads();
    if (threadIdx.x == 0) {
        best = red[0];
        for (int w = 1; w < (int)(blockDim.x >> 6); ++w) best = red[w] > best ? red[w] : best;
        const int idx = argmax_key_index(best);
        a.argmax_ws[m] = idx;
        if (a.argmax_out) a.argmax_out[m] = idx;
    }
    if (a.finish == FINISH_NONE) return;

    const int k = a.k_blk, b = m / k;
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        const unsigned prev = atomicAdd(&a.counters[b], 1u);
        s_last = (prev == (unsigned)k - 1) ? 1 : 0;
    }
    __syncthreads();
    if (!s_last || threadIdx.x != 0) return;
    __threadfence();
    const int32_t* am = a.argmax_ws + (size_t)b * k;
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
    __hip_atomic_store(&a.counters[b], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

hipError_t launch_argmax_finish(const ArgmaxArgs& a, hipStream_t s) {
    argmax_finish_kernel<<<a.M, 256, 0, s>>>(a);
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
