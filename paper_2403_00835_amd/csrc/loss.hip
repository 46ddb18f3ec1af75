// CLLM training loss head on gfx950: the global-consistency and AR losses of Section 3.2.2
// (eqs. global_loss, ar_loss) at the LM head, forward then backward.
//
// Inputs are LM-head input rows H (fp32): P teacher rows (conditioned on the fixed point y*,
// stop-gradient), P student rows (on the trajectory state y at the same positions) and A rows of
// the target model's generation with their target ids. The logits Z = H W^T come from the
// streaming GEMM (E_LOGITS epilogue). Per pair the loss is the forward KL D(p || q) between
// p = softmax(teacher logits) and q = softmax(student logits); per AR row -log softmax at the
// target; L = sum KL + omega sum NLL. Backward: D = dL/dZ for the student and AR rows
// (q - p; omega (softmax - onehot)), dH = D W (the streaming GEMM again, over a transposed copy
// of the packed LM head, K split across workgroups) and dW = D^T H (teacher rows get no
// gradient). In bf16 the fp32 operands D and H enter the MFMAs as hi + lo bf16 planes, as the
// activations of the forward do. Every sum has a fixed order (per-thread strided runs, fixed
// shuffle and wave trees, vocabulary chunks and K splits in index order), so results do not
// depend on timing.
#include <hip/hip_ext.h>

#include "device.h"
#include "launch.h"

namespace cllm {

namespace {

constexpr int kLossThreads = 256;
constexpr int kStat = 5;  // statistics per (row, chunk): pair (ma, za, cross, ms, zs); AR (mc, zc)

// Sum / max over a 256-thread workgroup in a fixed order (xor tree inside each wave, then the
// four waves in order); every thread gets the result.
template <bool MAX>
__device__ float block_reduce(float v, float *s_buf) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const float o = __shfl_xor(v, off);
        v = MAX ? fmaxf(v, o) : v + o;
    }
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) s_buf[w] = v;
    __syncthreads();
    return MAX ? fmaxf(fmaxf(s_buf[0], s_buf[1]), fmaxf(s_buf[2], s_buf[3]))
               : (s_buf[0] + s_buf[1]) + (s_buf[2] + s_buf[3]);
}

// Eight fp32 values as the hi and lo bf16 vectors of an MFMA operand (lo = bf16(x - hi)).
__device__ __forceinline__ void split8(const float (&x)[8], u32x4 &hi, u32x4 &lo) {
    uint32_t h[4], l[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint16_t h0 = f2bf(x[2 * i]), h1 = f2bf(x[2 * i + 1]);
        const uint16_t l0 = f2bf(x[2 * i] - bf2f(h0)), l1 = f2bf(x[2 * i + 1] - bf2f(h1));
        h[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        l[i] = (uint32_t)l0 | ((uint32_t)l1 << 16);
    }
    hi = u32x4{h[0], h[1], h[2], h[3]};
    lo = u32x4{l[0], l[1], l[2], l[3]};
}

// Operand order of an [n][r] matrix whose contraction index is r (rpad rows, zero past the
// data): for 16-row group n/16 and k-step r/32, lane 16 * ((r % 32) / 8) + n % 16, element r % 8.
__device__ __forceinline__ size_t tr_idx(int n, int r, int ks) {
    return ((size_t)((n >> 4) * ks + (r >> 5)) * kWave + 16 * ((r & 31) >> 3) + (n & 15)) * 8 + (r & 7);
}

}  // namespace

// Row statistics, phase 1: workgroup (chunk c of kLossChunk vocabulary entries, row item b); item
// b < P is pair b (teacher row b, student row P + b), item P + i is AR row i.
__global__ __launch_bounds__(kLossThreads) void loss_stats_kernel(LossParams p, float *stats, int nch) {
    __shared__ float s_buf[4];
    const int c = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    const int v0 = c * kLossChunk, v1 = min(v0 + kLossChunk, p.V);
    float *st = stats + ((size_t)b * nch + c) * kStat;
    if (b < p.P) {
        const float *a = p.Z + (size_t)b * p.ldz, *s = p.Z + (size_t)(p.P + b) * p.ldz;
        float ma = -INFINITY, ms = -INFINITY;
        for (int v = v0 + tid; v < v1; v += kLossThreads) {
            ma = fmaxf(ma, a[v]);
            ms = fmaxf(ms, s[v]);
        }
        ma = block_reduce<true>(ma, s_buf);
        ms = block_reduce<true>(ms, s_buf);
        float za = 0.f, zs = 0.f, cross = 0.f;
        for (int v = v0 + tid; v < v1; v += kLossThreads) {
            const float ea = expf(a[v] - ma);
            za += ea;
            zs += expf(s[v] - ms);
            cross += ea * (a[v] - s[v]);
        }
        za = block_reduce<false>(za, s_buf);
        zs = block_reduce<false>(zs, s_buf);
        cross = block_reduce<false>(cross, s_buf);
        if (tid == 0) {
            st[0] = ma;
            st[1] = za;
            st[2] = cross;
            st[3] = ms;
            st[4] = zs;
        }
    } else {
        const float *z = p.Z + (size_t)(2 * p.P + b - p.P) * p.ldz;
        float mc = -INFINITY;
        for (int v = v0 + tid; v < v1; v += kLossThreads) mc = fmaxf(mc, z[v]);
        mc = block_reduce<true>(mc, s_buf);
        float zc = 0.f;
        for (int v = v0 + tid; v < v1; v += kLossThreads) zc += expf(z[v] - mc);
        zc = block_reduce<false>(zc, s_buf);
        if (tid == 0) {
            st[0] = mc;
            st[1] = zc;
        }
    }
}

// Row statistics, phase 2: the chunks' statistics combined in chunk order (every thread the
// same), then the row's loss (chunk 0) and its logit gradients over the chunk (0 past V).
__global__ __launch_bounds__(kLossThreads) void loss_grad_kernel(LossParams p, const float *stats, int nch) {
    const int c = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    const int V = p.V, v0 = c * kLossChunk, v1 = min(v0 + kLossChunk, p.ldz);
    const float *st = stats + (size_t)b * nch * kStat;
    if (b < p.P) {
        float ma = -INFINITY, ms = -INFINITY;
        for (int q = 0; q < nch; ++q) {
            ma = fmaxf(ma, st[q * kStat + 0]);
            ms = fmaxf(ms, st[q * kStat + 3]);
        }
        float za = 0.f, zs = 0.f, cross = 0.f;
        for (int q = 0; q < nch; ++q) {
            const float fa = expf(st[q * kStat + 0] - ma);
            za += st[q * kStat + 1] * fa;
            cross += st[q * kStat + 2] * fa;
            zs += st[q * kStat + 4] * expf(st[q * kStat + 3] - ms);
        }
        // KL(p || q) = sum_v p_v (a_v - s_v) - logsumexp(a) + logsumexp(s)
        if (c == 0 && tid == 0) p.kl[b] = cross / za - (ma + logf(za)) + (ms + logf(zs));
        const float *a = p.Z + (size_t)b * p.ldz, *s = p.Z + (size_t)(p.P + b) * p.ldz;
        float *d = p.D + (size_t)b * p.ldz;
        const float ia = 1.0f / za, is = 1.0f / zs;
        for (int v = v0 + tid; v < v1; v += kLossThreads)
            d[v] = v < V ? expf(s[v] - ms) * is - expf(a[v] - ma) * ia : 0.0f;
    } else {
        const int i = b - p.P;
        const float *z = p.Z + (size_t)(2 * p.P + i) * p.ldz;
        const int t = p.targets[i];
        float *d = p.D + (size_t)(p.P + i) * p.ldz;
        if (t < 0 || t >= V) {  // a target outside the vocabulary: NaN loss and gradient row
            if (c == 0 && tid == 0) p.nll[i] = NAN;
            for (int v = v0 + tid; v < v1; v += kLossThreads) d[v] = v < V ? NAN : 0.0f;
            return;
        }
        float mc = -INFINITY;
        for (int q = 0; q < nch; ++q) mc = fmaxf(mc, st[q * kStat + 0]);
        float zc = 0.f;
        for (int q = 0; q < nch; ++q) zc += st[q * kStat + 1] * expf(st[q * kStat + 0] - mc);
        if (c == 0 && tid == 0) p.nll[i] = mc + logf(zc) - z[t];
        const float ic = 1.0f / zc;
        for (int v = v0 + tid; v < v1; v += kLossThreads)
            d[v] = v < V ? p.omega * (expf(z[v] - mc) * ic - (v == t ? 1.0f : 0.0f)) : 0.0f;
    }
}

// GEMM rows: teacher rows 0..np-1, student rows np..2np-1, AR rows 2np..2np+na-1.
template <Prec P>
__global__ void pack_rows_kernel(const float *T0, const float *S0, int np, const float *R0, int na, int d, int cap,
                                 void *A) {
    using T = typename PrecT<P>::T;
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (size_t)(2 * np + na) * d) return;
    const int r = (int)(i / d), k = (int)(i % d);
    const float x = r < np ? T0[(size_t)r * d + k] : r < 2 * np ? S0[(size_t)(r - np) * d + k]
                                                                 : R0[(size_t)(r - 2 * np) * d + k];
    put_act<P>(reinterpret_cast<T *>(A), act_plane(cap, d), act_idx<P>(r, k, d), x);
}

// Logit gradients D [rows][ldd] (fp32) as MFMA operands, bf16: thread (8 vocabulary entries, 8
// rows) writes the GEMM operand of dH = D W (rows r < rows, contraction over the vocabulary,
// Dact: two planes of cap rows x Vp) and the operand of dW = D^T H (contraction over the rows,
// DT: two planes of Vp x rpad, rows rows..rpad-1 zero).
__global__ __launch_bounds__(256) void pack_d_kernel(const float *D, int rows, int ldd, int Vp, int cap,
                                                     uint16_t *Dact, int rpad, uint16_t *DT) {
    const int nvb = Vp / 8;
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    const int vb = t % nvb, rb = t / nvb;
    if (rb * 8 >= rpad) return;
    const int v0 = vb * 8, r0 = rb * 8, ks = rpad / 32;
    float x[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int r = r0 + i;
        f32x4 lo4 = f32x4{0.f, 0.f, 0.f, 0.f}, hi4 = lo4;
        if (r < rows) {
            lo4 = *reinterpret_cast<const f32x4 *>(D + (size_t)r * ldd + v0);
            hi4 = *reinterpret_cast<const f32x4 *>(D + (size_t)r * ldd + v0 + 4);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            x[i][e] = lo4[e];
            x[i][4 + e] = hi4[e];
        }
    }
    const size_t pa = act_plane(cap, Vp), pt = (size_t)Vp * rpad;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        if (r0 + i >= rows) break;
        u32x4 h, l;
        split8(x[i], h, l);
        const size_t o = act_idx<Prec::BF16>(r0 + i, v0, Vp);  // 8 consecutive entries: one vector
        *reinterpret_cast<u32x4 *>(Dact + o) = h;
        *reinterpret_cast<u32x4 *>(Dact + pa + o) = l;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        float y[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) y[i] = x[i][j];
        u32x4 h, l;
        split8(y, h, l);
        const size_t o = tr_idx(v0 + j, r0, ks);
        *reinterpret_cast<u32x4 *>(DT + o) = h;
        *reinterpret_cast<u32x4 *>(DT + pt + o) = l;
    }
}

// fp32: the GEMM operand of dH = D W only (dW takes D as it is).
__global__ void pack_d_f32_kernel(const float *D, int rows, int ldd, int Vp, int cap, float *Dact) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (size_t)rows * Vp) return;
    const int r = (int)(i / Vp), v = (int)(i % Vp);
    Dact[act_idx<Prec::F32>(r, v, Vp)] = D[(size_t)r * ldd + v];
}

// Rows of dW = D^T H (student rows S0, then AR rows R0; zero from `rows` to rpad) as the bf16
// operand with contraction over the rows: HT, two planes of d x rpad. Thread: (column, 8 rows).
__global__ __launch_bounds__(256) void pack_ht_kernel(const float *S0, int np, const float *R0, int rows, int d,
                                                      int rpad, uint16_t *HT) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    const int k = t % d, rb = t / d;
    if (rb * 8 >= rpad) return;
    const int r0 = rb * 8;
    float x[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int r = r0 + i;
        x[i] = r >= rows ? 0.f : r < np ? S0[(size_t)r * d + k] : R0[(size_t)(r - np) * d + k];
    }
    u32x4 h, l;
    split8(x, h, l);
    const size_t o = tr_idx(k, r0, rpad / 32);
    *reinterpret_cast<u32x4 *>(HT + o) = h;
    *reinterpret_cast<u32x4 *>(HT + (size_t)d * rpad + o) = l;
}

// The packed LM head W [Vp][d] (tiles over (k-step of d, 16 vocabulary rows)) repacked as W^T
// [d][Vp] (tiles over (k-step of the vocabulary, 16 columns of d)), the weight operand of
// dH = D W. Thread: a VEC x VEC block (VEC vocabulary rows from v0, VEC columns from k0), read as
// VEC vectors along d and written as VEC vectors along the vocabulary.
template <Prec P>
__global__ __launch_bounds__(256) void transpose_lm_kernel(const uint8_t *W, int Vp, int d, uint8_t *WT) {
    using PT = PrecT<P>;
    using T = typename PT::T;
    constexpr int VEC = PT::VEC, KSTEP = PT::KSTEP;
    const int nvb = Vp / VEC;
    const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int vb = (int)(t % nvb), kb = (int)(t / nvb);
    if (kb >= d / VEC) return;
    const int v0 = vb * VEC, k0 = kb * VEC, Tv = Vp / 16, Td = d / 16;
    T x[VEC][VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
        const int v = v0 + i;
        const size_t tile = (size_t)(k0 / KSTEP) * Tv + v / 16;
        const int lane = 16 * ((k0 % KSTEP) / VEC) + v % 16;
        const u32x4 q = *reinterpret_cast<const u32x4 *>(W + tile * kTileBytes + (size_t)lane * 16);
        const T *e = reinterpret_cast<const T *>(&q);
#pragma unroll
        for (int j = 0; j < VEC; ++j) x[i][j] = e[j];
    }
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        const int k = k0 + j;
        const size_t tile = (size_t)(v0 / KSTEP) * Td + k / 16;
        const int lane = 16 * ((v0 % KSTEP) / VEC) + k % 16;
        alignas(16) T y[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) y[i] = x[i][j];
        *reinterpret_cast<u32x4 *>(WT + tile * kTileBytes + (size_t)lane * 16) = *reinterpret_cast<const u32x4 *>(y);
    }
}

// Sum of the K-split partials in split order; rows < np go to dS, the rest to dA.
__global__ void loss_dh_sum_kernel(const float *part, int nsplit, int n, int np_d, float *dS, float *dA) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (size_t)n) return;
    float s = 0.f;
    for (int c = 0; c < nsplit; ++c) s += part[(size_t)c * n + i];
    if (i < (size_t)np_d)
        dS[i] = s;
    else
        dA[i - np_d] = s;
}

// One workgroup per row: out = x (.) g / sqrt(mean(x^2) + eps), the LM head's input row.
__global__ __launch_bounds__(kLossThreads) void hidden_rows_kernel(const float *X, int ldx, int d, const float *g,
                                                                   float eps, float *out) {
    __shared__ float s_buf[4];
    const float *x = X + (size_t)blockIdx.x * ldx;
    float ss = 0.f;
    for (int k = threadIdx.x; k < d; k += kLossThreads) ss += x[k] * x[k];
    ss = block_reduce<false>(ss, s_buf);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
    for (int k = threadIdx.x; k < d; k += kLossThreads) out[(size_t)blockIdx.x * d + k] = x[k] * g[k] * inv;
}

// *loss = sum kl + omega * sum nll, each sum in row order, in double.
__global__ void loss_total_kernel(const float *kl, int np, const float *nll, int na, float omega, double *loss) {
    if (threadIdx.x != 0) return;
    double ks = 0.0, ns = 0.0;
    for (int i = 0; i < np; ++i) ks += (double)kl[i];
    for (int i = 0; i < na; ++i) ns += (double)nll[i];
    *loss = ks + (double)omega * ns;
}

// dW = D^T H, bf16 operands (hi + lo planes; the products hi hi + hi lo + lo hi, fp32
// accumulation). Workgroup: 128 vocabulary rows x 128 columns; wave (wv, wk) owns 64 x 64 (4 x 4
// tiles of 16 x 16); the contraction runs over the rpad rows, 32 per k-step. The wave's block
// goes out through LDS so that each store instruction writes four whole 256-byte row segments
// (16 bytes per lane) instead of 64-byte pieces of four rows.
constexpr int kDwV = 128, kDwK = 128, kDwLd = 64 + 4;  // LDS row stride (floats)
__global__ __launch_bounds__(256) void loss_dw_mfma_kernel(const uint16_t *DT, const uint16_t *HT, int Vp, int d,
                                                           int rpad, int V, float *dW) {
    __shared__ float s_blk[4][64 * kDwLd];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int nvt = Vp / 16, nkt = d / 16, ks = rpad / 32;
    // grid x: column blocks (fastest, so consecutive workgroups share the block of D^T through
    // L2), y: vocabulary blocks
    const int vt0 = blockIdx.y * (kDwV / 16) + (w & 1) * 4, kt0 = blockIdx.x * (kDwK / 16) + (w >> 1) * 4;
    const size_t pd = (size_t)Vp * rpad, ph = (size_t)d * rpad;
    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < ks; ++s) {
        u32x4 ah[4], al[4], bh[4], bl[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int vt = min(vt0 + i, nvt - 1);  // tiles past the end recompute the last (not stored)
            const size_t o = ((size_t)(vt * ks + s) * kWave + lane) * 8;
            ah[i] = *reinterpret_cast<const u32x4 *>(DT + o);
            al[i] = *reinterpret_cast<const u32x4 *>(DT + pd + o);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int kt = min(kt0 + j, nkt - 1);
            const size_t o = ((size_t)(kt * ks + s) * kWave + lane) * 8;
            bh[j] = *reinterpret_cast<const u32x4 *>(HT + o);
            bl[j] = *reinterpret_cast<const u32x4 *>(HT + ph + o);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                acc[i][j] = mfma_kstep<Prec::BF16>(ah[i], bh[j], acc[i][j]);
                acc[i][j] = mfma_kstep<Prec::BF16>(ah[i], bl[j], acc[i][j]);
                acc[i][j] = mfma_kstep<Prec::BF16>(al[i], bh[j], acc[i][j]);
            }
    }
    // C layout: row 4 * (lane / 16) + e of tile (i, j), column lane % 16; into the wave's LDS block
    float *blk = s_blk[w];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) blk[(16 * i + 4 * (lane >> 4) + e) * kDwLd + 16 * j + (lane & 15)] = acc[i][j][e];
    __syncthreads();
    // rows of the block: 16 lanes per row (16 bytes each), four rows per store
    const int k = 16 * kt0 + 4 * (lane & 15);
    if (k < d) {
#pragma unroll 4
        for (int r = lane >> 4; r < 64; r += 4) {
            const int v = 16 * vt0 + r;
            if (v < V) *reinterpret_cast<f32x4 *>(dW + (size_t)v * d + k) = *reinterpret_cast<const f32x4 *>(blk + r * kDwLd + 4 * (lane & 15));
        }
    }
}

// dW, fp32 operands: workgroup (64 vocabulary rows, 64 columns of d); wave w owns rows
// 16w..16w+15 and the 64 columns (four 16-column tiles); the sum runs over the gradient rows,
// 4 at a time.
__global__ __launch_bounds__(256) void loss_dw_f32_kernel(const float *D, int rows, int ldd, const float *S0, int np,
                                                          const float *R0, int d, int V, float *dW) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int v = blockIdx.x * 64 + 16 * w + (lane & 15), kb = blockIdx.y * 64;
    f32x4 acc[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) acc[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int r0 = 0; r0 < rows; r0 += 4) {
        const int r = r0 + (lane >> 4);
        const float a = (r < rows && v < V) ? D[(size_t)r * ldd + v] : 0.f;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
            const int k = kb + 16 * kt + (lane & 15);
            const float b = r >= rows ? 0.f : r < np ? S0[(size_t)r * d + k] : R0[(size_t)(r - np) * d + k];
            acc[kt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[kt], 0, 0, 0);
        }
    }
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int vo = blockIdx.x * 64 + 16 * w + 4 * (lane >> 4) + j;
            if (vo < V) dW[(size_t)vo * d + kb + 16 * kt + (lane & 15)] = acc[kt][j];
        }
}

hipError_t launch_loss_rows(const LossParams &p, float *stats, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    if (p.P < 0 || p.A < 0 || p.P + p.A < 1 || p.V < 1 || p.ldz < p.V) return hipErrorInvalidValue;
    const int nch = (p.ldz + kLossChunk - 1) / kLossChunk;  // = chunks of V (ldz - V < 64 <= kLossChunk)
    const dim3 grid(nch, p.P + p.A);
    if (e0)
        hipExtLaunchKernelGGL(loss_stats_kernel, grid, dim3(kLossThreads), 0, s, e0, nullptr, 0, p, stats, nch);
    else
        hipLaunchKernelGGL(loss_stats_kernel, grid, dim3(kLossThreads), 0, s, p, stats, nch);
    if (e1)
        hipExtLaunchKernelGGL(loss_grad_kernel, grid, dim3(kLossThreads), 0, s, nullptr, e1, 0, p,
                              (const float *)stats, nch);
    else
        hipLaunchKernelGGL(loss_grad_kernel, grid, dim3(kLossThreads), 0, s, p, (const float *)stats, nch);
    return hipGetLastError();
}

hipError_t launch_pack_rows(bool bf16, const float *T0, const float *S0, int np, const float *R0, int na, int d,
                            int cap, void *A, hipStream_t s, hipEvent_t e0) {
    const int rows = 2 * np + na;
    if (np < 0 || na < 0 || rows < 1 || rows > cap || d % 32 != 0) return hipErrorInvalidValue;
    const size_t n = (size_t)rows * d;
    const dim3 grid((unsigned)((n + 255) / 256));
    auto kern = bf16 ? pack_rows_kernel<Prec::BF16> : pack_rows_kernel<Prec::F32>;
    hipExtLaunchKernelGGL(kern, grid, dim3(256), 0, s, e0, nullptr, 0, T0, S0, np, R0, na, d, cap, A);
    return hipGetLastError();
}

hipError_t launch_loss_pack(bool bf16, const float *D, int rows, int ldd, int Vp, int cap, void *Dact, int rpad,
                            uint16_t *DT, const float *S0, int np, const float *R0, int d, uint16_t *HT,
                            hipStream_t s, hipEvent_t e1) {
    if (rows < 1 || rows > cap || ldd < Vp || Vp % 64 != 0 || d % 64 != 0) return hipErrorInvalidValue;
    if (!bf16) {
        const size_t n = (size_t)rows * Vp;
        hipExtLaunchKernelGGL(pack_d_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, nullptr, e1, 0,
                              D, rows, ldd, Vp, cap, reinterpret_cast<float *>(Dact));
        return hipGetLastError();
    }
    if (rpad % 32 != 0 || rpad < rows || rpad > cap || np < 0 || np > rows) return hipErrorInvalidValue;
    const size_t nd = (size_t)(Vp / 8) * (rpad / 8);
    hipLaunchKernelGGL(pack_d_kernel, dim3((unsigned)((nd + 255) / 256)), dim3(256), 0, s, D, rows, ldd, Vp, cap,
                       reinterpret_cast<uint16_t *>(Dact), rpad, DT);
    const size_t nh = (size_t)d * (rpad / 8);
    hipExtLaunchKernelGGL(pack_ht_kernel, dim3((unsigned)((nh + 255) / 256)), dim3(256), 0, s, nullptr, e1, 0, S0, np,
                          R0, rows, d, rpad, HT);
    return hipGetLastError();
}

hipError_t launch_transpose_lm(bool bf16, const uint8_t *W, int Vp, int d, uint8_t *WT, hipStream_t s) {
    if (Vp % 64 != 0 || d % 64 != 0) return hipErrorInvalidValue;
    const int vec = bf16 ? PrecT<Prec::BF16>::VEC : PrecT<Prec::F32>::VEC;
    const size_t n = (size_t)(Vp / vec) * (d / vec);
    const dim3 grid((unsigned)((n + 255) / 256));
    if (bf16)
        hipLaunchKernelGGL(transpose_lm_kernel<Prec::BF16>, grid, dim3(256), 0, s, W, Vp, d, WT);
    else
        hipLaunchKernelGGL(transpose_lm_kernel<Prec::F32>, grid, dim3(256), 0, s, W, Vp, d, WT);
    return hipGetLastError();
}

hipError_t launch_loss_dh_sum(const float *part, int nsplit, int rows, int d, int np, float *dS, float *dA,
                              hipStream_t s, hipEvent_t e1) {
    if (nsplit < 1 || rows < 1 || np < 0 || np > rows) return hipErrorInvalidValue;
    const int n = rows * d;
    hipExtLaunchKernelGGL(loss_dh_sum_kernel, dim3((n + 255) / 256), dim3(256), 0, s, nullptr, e1, 0, part, nsplit, n,
                          np * d, dS, dA);
    return hipGetLastError();
}

hipError_t launch_hidden_rows(const float *X, int ldx, int rows, int d, const float *g, float eps, float *out,
                              hipStream_t s) {
    if (rows < 1 || d < 1 || ldx < d) return hipErrorInvalidValue;
    hipLaunchKernelGGL(hidden_rows_kernel, dim3(rows), dim3(kLossThreads), 0, s, X, ldx, d, g, eps, out);
    return hipGetLastError();
}

hipError_t launch_loss_total(const float *kl, int np, const float *nll, int na, float omega, double *loss,
                             hipStream_t s) {
    hipLaunchKernelGGL(loss_total_kernel, dim3(1), dim3(64), 0, s, kl, np, nll, na, omega, loss);
    return hipGetLastError();
}

hipError_t launch_loss_dw(bool bf16, const uint16_t *DT, const uint16_t *HT, int Vp, int rpad, const float *D,
                          int rows, int ldd, const float *S0, int np, const float *R0, int d, int V, float *dW,
                          hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    if (rows < 1 || rows > 64 || np < 0 || np > rows || d % 64 != 0 || ldd < V || Vp < V || Vp % 64 != 0)
        return hipErrorInvalidValue;
    if (bf16) {
        if (rpad % 32 != 0 || rpad < rows) return hipErrorInvalidValue;
        const dim3 grid((d + kDwK - 1) / kDwK, (Vp + kDwV - 1) / kDwV);
        if (e0)
            hipExtLaunchKernelGGL(loss_dw_mfma_kernel, grid, dim3(256), 0, s, e0, e1, 0, DT, HT, Vp, d, rpad, V, dW);
        else
            hipLaunchKernelGGL(loss_dw_mfma_kernel, grid, dim3(256), 0, s, DT, HT, Vp, d, rpad, V, dW);
        return hipGetLastError();
    }
    const dim3 grid((V + 63) / 64, d / 64);
    if (e0)
        hipExtLaunchKernelGGL(loss_dw_f32_kernel, grid, dim3(256), 0, s, e0, e1, 0, D, rows, ldd, S0, np, R0, d, V, dW);
    else
        hipLaunchKernelGGL(loss_dw_f32_kernel, grid, dim3(256), 0, s, D, rows, ldd, S0, np, R0, d, V, dW);
    return hipGetLastError();
}

}  // namespace cllm
