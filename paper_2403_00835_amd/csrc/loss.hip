// CLLM training loss head on gfx950: the global-consistency and AR losses of Section 3.2.2
// (eqs. global_loss, ar_loss) at the LM head, forward then backward.
//
// Inputs are LM-head input rows H (fp32): P teacher rows (conditioned on the fixed point y*,
// stop-gradient), P student rows (on the trajectory state y at the same positions) and A rows of
// the target model's generation with their target ids. The logits Z = H W^T come from the
// streaming GEMM (E_LOGITS epilogue). Per pair the loss is the forward KL D(p || q) between
// p = softmax(teacher logits) and q = softmax(student logits); per AR row -log softmax at the
// target; L = sum KL + omega sum NLL. Backward: D = dL/dZ for the student and AR rows
// (q - p; omega (softmax - onehot)), dH = D W and dW = D^T H (teacher rows get no gradient).
// Every sum has a fixed order (per-thread strided runs, then fixed shuffle and wave trees; the
// vocabulary chunks of dH in chunk order), so results do not depend on timing.
#include <hip/hip_ext.h>

#include "device.h"
#include "launch.h"

namespace cllm {

namespace {

constexpr int kLossThreads = 256;

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

}  // namespace

// One workgroup per pair (blocks 0..P-1) or AR row (P..P+A-1).
__global__ __launch_bounds__(kLossThreads) void loss_rows_kernel(LossParams p) {
    __shared__ float s_buf[4];
    const int b = blockIdx.x, tid = threadIdx.x;
    const int V = p.V;
    if (b < p.P) {
        const float *a = p.Z + (size_t)b * p.ldz, *s = p.Z + (size_t)(p.P + b) * p.ldz;
        float ma = -INFINITY, ms = -INFINITY;
        for (int v = tid; v < V; v += kLossThreads) {
            ma = fmaxf(ma, a[v]);
            ms = fmaxf(ms, s[v]);
        }
        ma = block_reduce<true>(ma, s_buf);
        ms = block_reduce<true>(ms, s_buf);
        float za = 0.f, zs = 0.f, cross = 0.f;
        for (int v = tid; v < V; v += kLossThreads) {
            const float ea = expf(a[v] - ma);
            za += ea;
            zs += expf(s[v] - ms);
            cross += ea * (a[v] - s[v]);
        }
        za = block_reduce<false>(za, s_buf);
        zs = block_reduce<false>(zs, s_buf);
        cross = block_reduce<false>(cross, s_buf);
        // KL(p || q) = sum_v p_v (a_v - s_v) - logsumexp(a) + logsumexp(s)
        if (tid == 0) p.kl[b] = cross / za - (ma + logf(za)) + (ms + logf(zs));
        float *d = p.D + (size_t)b * p.ldz;
        const float ia = 1.0f / za, is = 1.0f / zs;
        for (int v = tid; v < p.ldz; v += kLossThreads)
            d[v] = v < V ? expf(s[v] - ms) * is - expf(a[v] - ma) * ia : 0.0f;
    } else {
        const int i = b - p.P;
        const float *c = p.Z + (size_t)(2 * p.P + i) * p.ldz;
        const int t = p.targets[i];
        float mc = -INFINITY;
        for (int v = tid; v < V; v += kLossThreads) mc = fmaxf(mc, c[v]);
        mc = block_reduce<true>(mc, s_buf);
        float zc = 0.f;
        for (int v = tid; v < V; v += kLossThreads) zc += expf(c[v] - mc);
        zc = block_reduce<false>(zc, s_buf);
        if (tid == 0) p.nll[i] = mc + logf(zc) - c[t];
        float *d = p.D + (size_t)(p.P + i) * p.ldz;
        const float ic = 1.0f / zc;
        for (int v = tid; v < p.ldz; v += kLossThreads)
            d[v] = v < V ? p.omega * (expf(c[v] - mc) * ic - (v == t ? 1.0f : 0.0f)) : 0.0f;
    }
}

template <Prec P>
__global__ void pack_rows_kernel(const float *X, int rows, int d, int cap, void *A) {
    using T = typename PrecT<P>::T;
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (size_t)rows * d) return;
    const int r = (int)(i / d), k = (int)(i % d);
    put_act<P>(reinterpret_cast<T *>(A), act_plane(cap, d), act_idx<P>(r, k, d), X[i]);
}

// dH partials: workgroup (64 columns of d, vocabulary chunk); 4 waves, wave w owns columns
// 16w..16w+15 for all rows (<= 64, four 16-row tiles). The chunk is taken 256 vocabulary rows at
// a time through LDS: W rows as fp32 [256][64] and D as [rows][256] (row stride 257).
constexpr int kDhSub = 256;

template <Prec P>
__global__ __launch_bounds__(256) void loss_dh_kernel(const float *D, int rows, int ldd, const uint8_t *W, int Vp,
                                                      int d, float *part) {
    using PT = PrecT<P>;
    using T = typename PT::T;
    __shared__ float s_w[kDhSub][64];
    __shared__ float s_d[64][kDhSub + 1];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int k0 = blockIdx.x * 64, chunk = blockIdx.y;
    const int T_ = Vp / 16;  // tiles per k-step
    f32x4 acc[4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int sub = 0; sub < kLossChunk / kDhSub; ++sub) {
        const int v0 = chunk * kLossChunk + sub * kDhSub;
        if (v0 >= Vp) break;
        // W rows v0..v0+255, columns k0..k0+63: element (v, k) sits in tile (k / KSTEP) * T_ + v / 16,
        // lane 16 * ((k % KSTEP) / VEC) + v % 16, element k % VEC.
        for (int e = tid; e < kDhSub * 64; e += 256) {
            const int vv = e / 64, kk = e % 64, v = v0 + vv, k = k0 + kk;
            float x = 0.f;
            if (v < Vp) {
                const size_t tile = (size_t)(k / PT::KSTEP) * T_ + v / 16;
                const int ln = 16 * ((k % PT::KSTEP) / PT::VEC) + v % 16;
                x = from_elem<P>(reinterpret_cast<const T *>(W + tile * kTileBytes)[ln * PT::VEC + k % PT::VEC]);
            }
            s_w[vv][kk] = x;
        }
        for (int e = tid; e < 64 * kDhSub; e += 256) {
            const int r = e / kDhSub, vv = e % kDhSub, v = v0 + vv;
            s_d[r][vv] = (r < rows && v < Vp) ? D[(size_t)r * ldd + v] : 0.f;
        }
        __syncthreads();
        for (int s4 = 0; s4 < kDhSub; s4 += 4) {
            const float bval = s_w[s4 + (lane >> 4)][16 * w + (lane & 15)];
#pragma unroll
            for (int rt = 0; rt < 4; ++rt)
                if (16 * rt < rows)
                    acc[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(s_d[16 * rt + (lane & 15)][s4 + (lane >> 4)], bval,
                                                                   acc[rt], 0, 0, 0);
        }
        __syncthreads();
    }
    // C layout: row 4 * (lane / 16) + j, column lane % 16
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 16 * rt + 4 * (lane >> 4) + j;
            if (r < rows) part[((size_t)chunk * rows + r) * d + k0 + 16 * w + (lane & 15)] = acc[rt][j];
        }
}

__global__ void loss_dh_sum_kernel(const float *part, int nch, int n, float *dH) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (size_t)n) return;
    float s = 0.f;
    for (int c = 0; c < nch; ++c) s += part[(size_t)c * n + i];  // chunk order
    dH[i] = s;
}

// dW: workgroup (64 vocabulary rows, 64 columns of d); wave w owns rows 16w..16w+15 and the 64
// columns (four 16-column tiles); the sum runs over the gradient rows, 4 at a time.
__global__ __launch_bounds__(256) void loss_dw_kernel(const float *D, int rows, int ldd, const float *H, int d, int V,
                                                      float *dW) {
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
            const float b = r < rows ? H[(size_t)r * d + kb + 16 * kt + (lane & 15)] : 0.f;
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

hipError_t launch_loss_rows(const LossParams &p, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    if (p.P < 0 || p.A < 0 || p.P + p.A < 1 || p.V < 1 || p.ldz < p.V) return hipErrorInvalidValue;
    if (e0)
        hipExtLaunchKernelGGL(loss_rows_kernel, dim3(p.P + p.A), dim3(kLossThreads), 0, s, e0, e1, 0, p);
    else
        hipLaunchKernelGGL(loss_rows_kernel, dim3(p.P + p.A), dim3(kLossThreads), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_pack_rows(bool bf16, const float *X, int rows, int d, int cap, void *A, hipStream_t s) {
    if (rows < 1 || rows > cap || d % 32 != 0) return hipErrorInvalidValue;
    const size_t n = (size_t)rows * d;
    const dim3 grid((unsigned)((n + 255) / 256));
    if (bf16)
        hipLaunchKernelGGL(pack_rows_kernel<Prec::BF16>, grid, dim3(256), 0, s, X, rows, d, cap, A);
    else
        hipLaunchKernelGGL(pack_rows_kernel<Prec::F32>, grid, dim3(256), 0, s, X, rows, d, cap, A);
    return hipGetLastError();
}

hipError_t launch_loss_dh(bool bf16, const float *D, int rows, int ldd, const uint8_t *W, int Vp, int d, float *part,
                          float *dH, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    if (rows < 1 || rows > 64 || d % 64 != 0 || Vp % 16 != 0 || ldd < Vp) return hipErrorInvalidValue;
    const int nch = (Vp + kLossChunk - 1) / kLossChunk;
    const dim3 grid(d / 64, nch);
    auto kern = bf16 ? loss_dh_kernel<Prec::BF16> : loss_dh_kernel<Prec::F32>;
    if (e0)
        hipExtLaunchKernelGGL(kern, grid, dim3(256), 0, s, e0, e1, 0, D, rows, ldd, W, Vp, d, part);
    else
        hipLaunchKernelGGL(kern, grid, dim3(256), 0, s, D, rows, ldd, W, Vp, d, part);
    const int n = rows * d;
    hipLaunchKernelGGL(loss_dh_sum_kernel, dim3((n + 255) / 256), dim3(256), 0, s, part, nch, n, dH);
    return hipGetLastError();
}

hipError_t launch_loss_dw(const float *D, int rows, int ldd, const float *H, int d, int V, float *dW, hipStream_t s,
                          hipEvent_t e0, hipEvent_t e1) {
    if (rows < 1 || rows > 64 || d % 64 != 0 || ldd < V) return hipErrorInvalidValue;
    const dim3 grid((V + 63) / 64, d / 64);
    if (e0)
        hipExtLaunchKernelGGL(loss_dw_kernel, grid, dim3(256), 0, s, e0, e1, 0, D, rows, ldd, H, d, V, dW);
    else
        hipLaunchKernelGGL(loss_dw_kernel, grid, dim3(256), 0, s, D, rows, ldd, H, d, V, dW);
    return hipGetLastError();
}

}  // namespace cllm
