// HIP kernels of one Jacobi iteration on gfx950 (CDNA4).
//
// An iteration over a block of m tokens at positions L .. L+m-1 (Section 3.1: one causal forward
// pass over the n-token block gives all n greedy predictions) is the launch sequence
//   embed -> per layer [QKV GEMM (+RMSNorm prologue, +RoPE, +provisional KV write)
//                       -> attention partials -> attention combine
//                       -> O GEMM (+residual) -> gate/up GEMM (+RMSNorm prologue, +SwiGLU)
//                       -> down GEMM (+residual)]
//   -> LM-head GEMM (+RMSNorm prologue, +argmax partials) -> scan/commit.
// Every kernel reads m and L from the device control block, so the same sequence serves every
// iteration without host round trips.
//
// Determinism: every reduction has a fixed order that depends only on the model shape, never on
// m, so a row's results do not depend on how many rows are in the block. Hence greedy decoding
// with blocks of one token (AR) and Jacobi decoding produce bit-identical tokens.
#include <hip/hip_ext.h>

#include "device.h"
#include "launch.h"

namespace cllm {

// ------------------------------------------------------------------------------------------
// Weight-streaming GEMM:  Y[rows x N] = A[rows x K] * W^T,  W packed in 1 KiB tiles.
//
// Packed layout: tile (t, s) covers weight rows 16t .. 16t+15 (after the per-GEMM row order)
// and K indices s*KSTEP .. s*KSTEP+KSTEP-1; lane l's 16 bytes are row 16t + l%16, K indices
// s*KSTEP + (l/16)*VEC .. +VEC. Tiles of one row block are contiguous over s.
//
// A workgroup of 8 waves owns NT consecutive tiles (16*NT output columns) for all rows; wave w
// takes k-steps w, w+8, w+16, ... and accumulates them in order with MFMA; the 8 partial tiles
// are then summed in a fixed tree ((w0+w4)+(w2+w6))+((w1+w5)+(w3+w7)). Weights are read once,
// straight into registers (no LDS); the activation rows (a few KiB, L2-resident) are re-read.
// ------------------------------------------------------------------------------------------

enum ALoad { A_ACT = 0, A_NORM = 1 };
enum Epi { E_QKV = 0, E_RESID = 1, E_SWIGLU = 2, E_ARGMAX = 3 };

template <Prec P, int RG>
struct ARaw;
template <int RG>
struct ARaw<Prec::BF16, RG> {  // norm loader keeps 8 fp32 values per row group
    u32x4 lo[RG], hi[RG];
};
template <int RG>
struct ARaw<Prec::F32, RG> {
    u32x4 lo[RG];
};

template <Prec P, int NT, int RG, int AL>
struct Stage {
    u32x4 b[2][NT];            // two k-steps per stage
    u32x4 a[2][RG];            // activation operand (A_ACT)
    ARaw<P, RG> x[2];          // raw fp32 rows (A_NORM)
};

template <Prec P, int NT, int RG, int AL>
__device__ __forceinline__ void gemm_load(Stage<P, NT, RG, AL> &st, const GemmParams &p, int t0, int base,
                                          int lane) {
    using PT = PrecT<P>;
    const int g = lane >> 4, r16 = lane & 15;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int s = base + u * kGemmWaves;
        if (s < p.Ks) {
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                const u32x4 *src = reinterpret_cast<const u32x4 *>(p.W + ((size_t)(t0 + j) * p.Ks + s) * kTileBytes) + lane;
                st.b[u][j] = __builtin_nontemporal_load(src);
            }
            const int k = s * PT::KSTEP + g * PT::VEC;
            if constexpr (AL == A_ACT) {
                using T = typename PT::T;
                const T *A = reinterpret_cast<const T *>(p.A);
#pragma unroll
                for (int r = 0; r < RG; ++r)
                    st.a[u][r] = *reinterpret_cast<const u32x4 *>(A + (size_t)(16 * r + r16) * p.lda + k);
            } else {
#pragma unroll
                for (int r = 0; r < RG; ++r) {
                    const float *xr = p.X + (size_t)(16 * r + r16) * p.ldx + k;
                    st.x[u].lo[r] = *reinterpret_cast<const u32x4 *>(xr);
                    if constexpr (P == Prec::BF16) st.x[u].hi[r] = *reinterpret_cast<const u32x4 *>(xr + 4);
                }
            }
        }
    }
}

template <Prec P, int NT, int RG, int AL>
__device__ __forceinline__ void gemm_compute(const Stage<P, NT, RG, AL> &st, const GemmParams &p, int base,
                                             int lane, f32x4 (&acc)[RG][NT], const float *s_inv,
                                             const float *s_gain) {
    using PT = PrecT<P>;
    const int g = lane >> 4, r16 = lane & 15;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int s = base + u * kGemmWaves;
        if (s < p.Ks) {
#pragma unroll
            for (int r = 0; r < RG; ++r) {
                u32x4 a;
                if constexpr (AL == A_ACT) {
                    a = st.a[u][r];
                } else {
                    const int k = s * PT::KSTEP + g * PT::VEC;
                    const float inv = s_inv[16 * r + r16];
                    const float *gk = s_gain + k;
                    if constexpr (P == Prec::BF16) {
                        const u32x4 lo = st.x[u].lo[r], hi = st.x[u].hi[r];
                        float v[8] = {__uint_as_float(lo.x), __uint_as_float(lo.y), __uint_as_float(lo.z),
                                      __uint_as_float(lo.w), __uint_as_float(hi.x), __uint_as_float(hi.y),
                                      __uint_as_float(hi.z), __uint_as_float(hi.w)};
                        uint32_t w[4];
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            uint32_t e0 = f2bf(v[2 * q] * inv * gk[2 * q]);
                            uint32_t e1 = f2bf(v[2 * q + 1] * inv * gk[2 * q + 1]);
                            w[q] = e0 | (e1 << 16);
                        }
                        a = u32x4{w[0], w[1], w[2], w[3]};
                    } else {
                        const u32x4 lo = st.x[u].lo[r];
                        a = u32x4{__float_as_uint(__uint_as_float(lo.x) * inv * gk[0]),
                                  __float_as_uint(__uint_as_float(lo.y) * inv * gk[1]),
                                  __float_as_uint(__uint_as_float(lo.z) * inv * gk[2]),
                                  __float_as_uint(__uint_as_float(lo.w) * inv * gk[3])};
                    }
                }
#pragma unroll
                for (int j = 0; j < NT; ++j) acc[r][j] = mfma_kstep<P>(a, st.b[u][j], acc[r][j]);
            }
        }
    }
}

__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

template <Prec P, int NT, int RG, int AL, int EP>
__global__ __launch_bounds__(kGemmWaves * kWave) void gemm_kernel(GemmParams p) {
    using PT = PrecT<P>;
    using T = typename PT::T;
    const Ctl *ctl = p.ctl;
    const int m = ctl->m;
    if (m <= 0) return;
    const int L = ctl->L;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int wg = blockIdx.x;
    const int t0 = wg * NT;
    constexpr int ROWS = 16 * RG, COLS = 16 * NT;

    extern __shared__ float smem[];
    float *s_red = smem;                          // 4 x NT x 64 x 4 (also ROWS x 16 for E_RESID)
    float *s_tile = s_red + 4 * NT * 256;         // ROWS x (COLS + 1)
    float *s_inv = s_tile + ROWS * (COLS + 1);    // ROWS
    float *s_gain = s_inv + kMaxRows;             // K (A_NORM only)

    if constexpr (AL == A_NORM) {
        for (int k = tid; k < p.K; k += kGemmWaves * kWave) s_gain[k] = p.gain[k];
        // Row factor 1/sqrt(mean(x^2) + eps) from the producer's per-16-column partial sums:
        // 8 threads per row sum strided partials in order, then a fixed xor tree.
        if (tid < ROWS * 8) {
            const int row = tid >> 3, part = tid & 7;
            float sum = 0.0f;
            for (int t = part; t < p.T; t += 8) sum += p.ssq[(size_t)t * kMaxRows + row];
            sum += __shfl_xor(sum, 4, 8);
            sum += __shfl_xor(sum, 2, 8);
            sum += __shfl_xor(sum, 1, 8);
            if (part == 0) s_inv[row] = 1.0f / sqrtf(sum / (float)p.K + p.eps);
        }
        __syncthreads();
    }

    f32x4 acc[RG][NT];
#pragma unroll
    for (int r = 0; r < RG; ++r)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[r][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Two-stage software pipeline over this wave's k-steps (each stage = 2 k-steps).
    {
        Stage<P, NT, RG, AL> s0, s1;
        int base = w;
        gemm_load(s0, p, t0, base, lane);
        while (true) {
            int nb = base + 2 * kGemmWaves;
            if (nb < p.Ks) gemm_load(s1, p, t0, nb, lane);
            gemm_compute(s0, p, base, lane, acc, s_inv, s_gain);
            if (nb >= p.Ks) break;
            base = nb;
            nb = base + 2 * kGemmWaves;
            if (nb < p.Ks) gemm_load(s0, p, t0, nb, lane);
            gemm_compute(s1, p, base, lane, acc, s_inv, s_gain);
            if (nb >= p.Ks) break;
            base = nb;
        }
    }

    // Fixed-tree reduction of the 8 waves' partial tiles through LDS, one row group at a time:
    // ((w0+w4)+(w2+w6))+((w1+w5)+(w3+w7)) for every element.
#pragma unroll
    for (int r = 0; r < RG; ++r) {
#pragma unroll
        for (int half = 4; half >= 1; half >>= 1) {
            if (w >= half && w < 2 * half) {
                float *dst = s_red + (size_t)(w - half) * NT * 256;
#pragma unroll
                for (int j = 0; j < NT; ++j) *reinterpret_cast<f32x4 *>(dst + (j * 64 + lane) * 4) = acc[r][j];
            }
            __syncthreads();
            if (w < half) {
                const float *src = s_red + (size_t)w * NT * 256;
#pragma unroll
                for (int j = 0; j < NT; ++j) acc[r][j] += *reinterpret_cast<const f32x4 *>(src + (j * 64 + lane) * 4);
            }
            __syncthreads();
        }
        if (w == 0) {
            // C layout of a 16x16 MFMA tile: lane l holds rows 4*(l/16)+v, column l%16.
#pragma unroll
            for (int j = 0; j < NT; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    s_tile[(16 * r + 4 * (lane >> 4) + v) * (COLS + 1) + 16 * j + (lane & 15)] = acc[r][j][v];
        }
    }
    __syncthreads();

    // ---------------------------------------------------------------- epilogues
    if constexpr (EP == E_QKV) {
        // Packed columns -> (section, head, dim). With head_dim >= 32 a workgroup's two tiles are
        // dims [16b, 16b+16) and [hd/2+16b, hd/2+16b+16) of one head (rotate-half partners);
        // with head_dim 16 one tile is a whole head.
        const int hd = p.hd, d = p.d, h2 = hd >> 1;
        for (int idx = tid; idx < ROWS * COLS; idx += kGemmWaves * kWave) {
            const int row = idx / COLS, pc = idx % COLS;
            if (row >= m) continue;
            const int R = t0 * 16 + pc;  // packed row index
            int sec, head, dim, partner;
            if (hd >= 32) {
                const int per_sec = d;  // packed rows per section
                sec = R / per_sec;
                const int within = R % per_sec;
                head = within / hd;
                const int q = within % hd, b16 = q >> 4, o = q & 15;
                dim = (b16 & 1) ? (h2 + (b16 >> 1) * 16 + o) : ((b16 >> 1) * 16 + o);
                partner = pc ^ 16;
            } else {
                sec = R / d;
                head = (R % d) / hd;
                dim = R % hd;
                partner = pc ^ h2;
            }
            const int pos = L + row;
            float x = s_tile[row * (COLS + 1) + pc];
            if (sec < 2) {
                const float y = s_tile[row * (COLS + 1) + partner];
                const int j = dim < h2 ? dim : dim - h2;
                const float c = p.rcos[(size_t)pos * h2 + j], s = p.rsin[(size_t)pos * h2 + j];
                x = dim < h2 ? (x * c - y * s) : (x * c + y * s);
            }
            const T e = to_elem<P>(x);
            const int col = head * hd + dim;
            if (sec == 0)
                reinterpret_cast<T *>(p.Q)[(size_t)row * d + col] = e;
            else if (sec == 1)
                reinterpret_cast<T *>(p.Kc)[(size_t)pos * d + col] = e;
            else
                reinterpret_cast<T *>(p.Vt)[(size_t)col * p.ctx_alloc + pos] = e;
        }
    } else if constexpr (EP == E_RESID) {
        static_assert(NT == 1, "residual epilogue owns one 16-column tile");
        const int c0 = t0 * 16;
        float *s_sq = s_red;  // reuse: ROWS x 16
        for (int idx = tid; idx < ROWS * 16; idx += kGemmWaves * kWave) {
            const int row = idx >> 4, c = idx & 15;
            float v = 0.0f;
            if (row < m) {
                float *xp = p.Xout + (size_t)row * p.ldx + c0 + c;
                v = *xp + s_tile[row * (COLS + 1) + c];
                *xp = v;
            }
            s_sq[idx] = v * v;
        }
        __syncthreads();
        if (tid < ROWS && tid < m) {
            float sum = 0.0f;
#pragma unroll
            for (int c = 0; c < 16; ++c) sum += s_sq[tid * 16 + c];
            p.ssq_out[(size_t)t0 * kMaxRows + tid] = sum;
        }
    } else if constexpr (EP == E_SWIGLU) {
        static_assert(NT == 2, "gate/up epilogue pairs a gate tile with an up tile");
        for (int idx = tid; idx < ROWS * 16; idx += kGemmWaves * kWave) {
            const int row = idx >> 4, c = idx & 15;
            if (row >= m) continue;
            const float gt = s_tile[row * (COLS + 1) + c];
            const float up = s_tile[row * (COLS + 1) + 16 + c];
            reinterpret_cast<T *>(p.H)[(size_t)row * p.Fp + wg * 16 + c] = to_elem<P>(silu(gt) * up);
        }
    } else {  // E_ARGMAX
        // One wave per row: (max, lowest column) over this workgroup's columns < V.
        for (int row = w; row < ROWS; row += kGemmWaves) {
            if (row >= m) break;
            float bv = -INFINITY;
            int bi = 0x7fffffff;
            int nan = 0;
            for (int c = lane; c < COLS; c += kWave) {
                const int col = t0 * 16 + c;
                if (col < p.V) {
                    const float v = s_tile[row * (COLS + 1) + c];
                    if (p.dbg) p.dbg[(size_t)row * p.V + col] = v;
                    if (v != v) nan = 1;
                    else if (v > bv || (v == bv && col < bi)) { bv = v; bi = col; }
                }
            }
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) {
                const float ov = __shfl_xor(bv, off);
                const int oi = __shfl_xor(bi, off);
                nan |= __shfl_xor(nan, off);
                if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
            }
            if (lane == 0) {
                p.pmax[(size_t)wg * kMaxRows + row] = bv;
                p.pidx[(size_t)wg * kMaxRows + row] = nan ? -1 : bi;
            }
        }
    }
}

// ------------------------------------------------------------------------------------------
// Embedding gather: X[i] = E[z_i] (fp32) and the per-16-column sums of squares for the first
// RMSNorm.
// ------------------------------------------------------------------------------------------
template <Prec P>
__global__ __launch_bounds__(256) void embed_kernel(EmbedParams p) {
    using T = typename PrecT<P>::T;
    const Ctl *ctl = p.ctl;
    const int m = ctl->m;
    const int row = blockIdx.x;
    if (row >= m) return;
    const int tok = ctl->z[row];
    const T *e = reinterpret_cast<const T *>(p.E) + (size_t)tok * p.d;
    float *x = p.X + (size_t)row * p.d;
    for (int t = threadIdx.x; t < p.d / 16; t += blockDim.x) {
        float sum = 0.0f;
#pragma unroll
        for (int c = 0; c < 16; ++c) {
            const float v = from_elem<P>(e[16 * t + c]);
            x[16 * t + c] = v;
            sum += v * v;
        }
        p.ssq[(size_t)t * kMaxRows + row] = sum;
    }
}

// ------------------------------------------------------------------------------------------
// Block-causal attention, split over fixed 64-key chunks at absolute positions.
// Workgroup (chunk c, head h), one wave per 16 query rows. With the cache K [pos][d] and the
// transposed value cache Vt [d][pos]:
//   S^T = K_chunk * Q^T   (MFMA A operand = key rows, B operand = query rows)
//   softmax over keys j <= L + i (fp32, base-2 exponent with the 1/sqrt(hd) scale folded in)
//   O^T = Vt_chunk * P^T  (the lane's own S^T registers are the B operand; the V^T loads use
//                          the same K-slot assignment)
// Each (h, c, row) writes a partial (max, sum, unnormalised output).
// ------------------------------------------------------------------------------------------
template <Prec P, int RG>
__global__ __launch_bounds__(kWave * RG) void attn_partial_kernel(AttnParams p) {
    using PT = PrecT<P>;
    using T = typename PT::T;
    const Ctl *ctl = p.ctl;
    const int m = ctl->m;
    if (m <= 0) return;
    const int L = ctl->L;
    const int c = blockIdx.x, h = blockIdx.y;
    const int key0 = c * kAttnChunk;
    if (key0 >= L + m) return;  // no key of this chunk is visible to any row
    const int lane = threadIdx.x & 63, rg = threadIdx.x >> 6;
    const int g = lane >> 4, r16 = lane & 15;
    const int hd = p.hd, d = p.d;
    const int qrow = 16 * rg + r16;
    const int qpos = L + qrow;
    const T *Kc = reinterpret_cast<const T *>(p.Kc);
    const T *Vt = reinterpret_cast<const T *>(p.Vt);
    const T *Q = reinterpret_cast<const T *>(p.Q);

    f32x4 st[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) st[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int kk = 0; kk < hd / PT::KSTEP; ++kk) {
        const int dcol = h * hd + kk * PT::KSTEP + g * PT::VEC;
        const u32x4 qv = *reinterpret_cast<const u32x4 *>(Q + (size_t)qrow * d + dcol);
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
            const u32x4 kv = *reinterpret_cast<const u32x4 *>(Kc + (size_t)(key0 + 16 * kt + r16) * d + dcol);
            st[kt] = mfma_kstep<P>(kv, qv, st[kt]);
        }
    }
    // st[kt][v] = S^T[key0 + 16kt + 4g + v][qrow]
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int key = key0 + 16 * kt + 4 * g + v;
            const float s = key <= qpos ? st[kt][v] * p.scale_log2 : -INFINITY;
            st[kt][v] = s;
            mx = fmaxf(mx, s);
        }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    float l = 0.0f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            float pr = (mx == -INFINITY || st[kt][v] == -INFINITY) ? 0.0f : exp2f(st[kt][v] - mx);
            if constexpr (P == Prec::BF16) pr = bf2f(f2bf(pr));  // the PV product consumes bf16
            st[kt][v] = pr;
            l += pr;
        }
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);

    const size_t pbase = ((size_t)h * p.nch + c) * kMaxRows + qrow;
    for (int dt = 0; dt < hd / 16; ++dt) {
        const T *vrow = Vt + (size_t)(h * hd + 16 * dt + r16) * p.ctx_alloc + key0;
        f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
        if constexpr (P == Prec::BF16) {
#pragma unroll
            for (int kp = 0; kp < 2; ++kp) {
                // K slots: keys 32kp + 4g + (0..3) and 32kp + 16 + 4g + (0..3).
                const u32x2 va = *reinterpret_cast<const u32x2 *>(vrow + 32 * kp + 4 * g);
                const u32x2 vb = *reinterpret_cast<const u32x2 *>(vrow + 32 * kp + 16 + 4 * g);
                const f32x4 pa = st[2 * kp], pb = st[2 * kp + 1];
                const u32x4 bop = u32x4{(uint32_t)f2bf(pa[0]) | ((uint32_t)f2bf(pa[1]) << 16),
                                        (uint32_t)f2bf(pa[2]) | ((uint32_t)f2bf(pa[3]) << 16),
                                        (uint32_t)f2bf(pb[0]) | ((uint32_t)f2bf(pb[1]) << 16),
                                        (uint32_t)f2bf(pb[2]) | ((uint32_t)f2bf(pb[3]) << 16)};
                o = mfma_kstep<P>(u32x4{va.x, va.y, vb.x, vb.y}, bop, o);
            }
        } else {
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) {
                const u32x4 va = *reinterpret_cast<const u32x4 *>(vrow + 16 * kt + 4 * g);
                const f32x4 pk = st[kt];
                o = mfma_kstep<P>(va, u32x4{__float_as_uint(pk[0]), __float_as_uint(pk[1]), __float_as_uint(pk[2]),
                                            __float_as_uint(pk[3])},
                                  o);
            }
        }
        // o[v] = O^T[16dt + 4g + v][qrow]
        *reinterpret_cast<f32x4 *>(p.Opart + pbase * hd + 16 * dt + 4 * g) = o;
    }
    if (g == 0) {
        p.Mpart[pbase] = mx;
        p.Lpart[pbase] = l;
    }
}

// Combine the chunk partials of one (head, row) in chunk order and write bf16/fp32 O.
template <Prec P>
__global__ void attn_combine_kernel(AttnParams p) {
    using T = typename PrecT<P>::T;
    const Ctl *ctl = p.ctl;
    const int m = ctl->m;
    const int h = blockIdx.x, row = blockIdx.y;
    if (row >= m) return;
    const int L = ctl->L;
    const int nlive = (L + m + kAttnChunk - 1) / kAttnChunk;
    const int dim = threadIdx.x;
    const size_t b0 = (size_t)h * p.nch * kMaxRows + row;
    float M = -INFINITY;
    for (int c = 0; c < nlive; ++c) M = fmaxf(M, p.Mpart[b0 + (size_t)c * kMaxRows]);
    float den = 0.0f, num = 0.0f;
    for (int c = 0; c < nlive; ++c) {
        const size_t b = b0 + (size_t)c * kMaxRows;
        const float mc = p.Mpart[b];
        const float wc = mc == -INFINITY ? 0.0f : exp2f(mc - M);
        den += wc * p.Lpart[b];
        num += wc * p.Opart[b * p.hd + dim];
    }
    reinterpret_cast<T *>(p.O)[(size_t)row * p.d + h * p.hd + dim] = to_elem<P>(num / den);
}

// ------------------------------------------------------------------------------------------
// Scan / commit (one wave): final argmax over the LM-head workgroups (in column order, ties to
// the lowest id), accepted length a = 1 + leading matches z[k] == pred[k-1], commit L += a,
// emit z[0..a), pending = pred[a-1], and in decode mode the next block.
// ------------------------------------------------------------------------------------------
__device__ int32_t draw_guess(const Ctl *c, const int32_t *stream, int32_t t, int32_t d) {
    const uint64_t h = mix64(mix64(mix64(mix64(c->seed) ^ (uint64_t)(uint32_t)c->seq) ^ (uint64_t)(uint32_t)t) ^
                             (uint64_t)(uint32_t)d);
    const uint64_t V = (uint64_t)(uint32_t)c->vocab;
    if (c->policy == 0 || stream == nullptr) return (int32_t)(((h >> 32) * V) >> 32);
    const int32_t s = t < c->stream_len ? stream[t] : 0;
    if ((h >> 11) < c->thr53) {
        const uint64_t h2 = mix64(h);
        const int32_t r = (int32_t)(((h2 >> 32) * (V - 1)) >> 32);
        return (int32_t)(((int64_t)s + 1 + r) % (int64_t)V);
    }
    return s;
}

// Lay out the first block of a decode after the prefill.
__global__ void decode_init_kernel(ScanParams p) {
    Ctl *c = p.ctl;
    if (threadIdx.x != 0) return;
    c->mode = MODE_DECODE;
    c->e = 0;
    c->b0 = 0;
    c->nb = c->n < c->max_new ? c->n : c->max_new;
    c->steps = 0;
    c->blocks = 1;
    c->done = 0;
    c->err = 0;
    for (int i = 0; i <= kMaxBlock; ++i) c->hist[i] = 0;
    c->z[0] = c->pending;
    for (int j = 1; j < c->nb; ++j) c->z[j] = draw_guess(c, p.stream, j, 0);
    c->m = c->nb;
}

__global__ __launch_bounds__(kWave) void scan_commit_kernel(ScanParams p) {
    Ctl *c = p.ctl;
    const int m = c->m;
    if (m <= 0) return;
    const int lane = threadIdx.x;
    if (p.advance_only) {
        if (lane == 0) {
            c->L += m;
            c->m = 0;
        }
        return;
    }
    if (lane < m) {
        float bv = -INFINITY;
        int bi = -2;
        for (int g = 0; g < p.n_wg; ++g) {
            const int idx = p.pidx[(size_t)g * kMaxRows + lane];
            const float v = p.pmax[(size_t)g * kMaxRows + lane];
            if (idx < 0) { bi = -1; break; }
            if (bi == -2 || v > bv) { bv = v; bi = idx; }
        }
        c->pred[lane] = bi;
    }
    __syncthreads();
    if (lane != 0) return;
    for (int i = 0; i < m; ++i)
        if (c->pred[i] < 0) {
            c->err |= 1;
            c->done = 1;
            c->m = 0;
            return;
        }
    if (c->mode == MODE_PREFILL) {
        c->L += m;
        c->pending = c->pred[m - 1];
        c->m = 0;
        return;
    }
    int a = 1;
    while (a < m && c->z[a] == c->pred[a - 1]) ++a;
    c->L += a;
    c->a_last = a;
    c->steps += 1;
    c->hist[a] += 1;
    c->pending = c->pred[a - 1];
    if (c->mode != MODE_DECODE) {
        c->m = 0;
        return;
    }
    for (int k = 0; k < a; ++k) p.out[c->e + k] = c->z[k];
    c->e += a;
    if (c->e >= c->max_new) {
        c->done = 1;
        c->m = 0;
        return;
    }
    const int e = c->e, n = c->n;
    const int draw = c->policy == 2 ? c->steps : 0;
    int newm;
    if (c->block_policy == 0) {
        if (e == c->b0 + c->nb) {  // block converged; its last prediction seeds the next block
            c->b0 = e;
            c->nb = (c->max_new - e) < n ? (c->max_new - e) : n;
            c->blocks += 1;
            newm = c->nb;
            for (int j = 1; j < newm; ++j) c->z[j] = draw_guess(c, p.stream, e + j, draw);
        } else {
            newm = c->b0 + c->nb - e;
            for (int j = 1; j < newm; ++j)
                c->z[j] = c->policy == 2 ? draw_guess(c, p.stream, e + j, draw) : c->pred[a - 1 + j];
        }
    } else {
        newm = (c->max_new - e) < n ? (c->max_new - e) : n;
        for (int j = 1; j < newm; ++j) {
            const int src = a - 1 + j;
            c->z[j] = (c->policy != 2 && src < m) ? c->pred[src] : draw_guess(c, p.stream, e + j, draw);
        }
    }
    c->z[0] = c->pending;
    c->m = newm;
}

// ------------------------------------------------------------------------------------------
// Weight repacking into the streaming tile layout. perm[r] is the logical source row of packed
// row r (-1: zero padding).
// ------------------------------------------------------------------------------------------
template <Prec P>
__global__ void repack_kernel(const void *src, const int32_t *perm, int K, int Ks, int n_tiles, uint8_t *dst) {
    using PT = PrecT<P>;
    using T = typename PT::T;
    const size_t tile = (size_t)blockIdx.x + (size_t)blockIdx.y * gridDim.x;
    if (tile >= (size_t)n_tiles * Ks) return;
    const int t = (int)(tile / Ks), s = (int)(tile % Ks);
    const int lane = threadIdx.x, g = lane >> 4, r16 = lane & 15;
    const int row = perm[16 * t + r16];
    T v[PT::VEC];
#pragma unroll
    for (int e = 0; e < PT::VEC; ++e) {
        const int k = s * PT::KSTEP + g * PT::VEC + e;
        v[e] = (row >= 0 && k < K) ? reinterpret_cast<const T *>(src)[(size_t)row * K + k] : T(0);
    }
    T *out = reinterpret_cast<T *>(dst + tile * kTileBytes) + lane * PT::VEC;
#pragma unroll
    for (int e = 0; e < PT::VEC; ++e) out[e] = v[e];
}

// ------------------------------------------------------------------------------------------
// Launchers
// ------------------------------------------------------------------------------------------
template <Prec P, int NT, int RG, int AL, int EP>
static hipError_t launch_gemm_t(const GemmParams &p, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    constexpr int ROWS = 16 * RG, COLS = 16 * NT;
    static_assert(4 * NT * 256 >= ROWS * 16, "E_RESID reuses the reduction buffer");
    size_t lds = (size_t)(4 * NT * 256 + ROWS * (COLS + 1) + kMaxRows) * sizeof(float);
    if (AL == A_NORM) lds += (size_t)p.K * sizeof(float);
    auto kern = gemm_kernel<P, NT, RG, AL, EP>;
    if (lds > 64 * 1024) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (err != hipSuccess) return err;
    }
    if (e0) {
        hipExtLaunchKernelGGL(kern, dim3(p.n_wg), dim3(kGemmWaves * kWave), lds, s, e0, e1, 0, p);
    } else {
        hipLaunchKernelGGL(kern, dim3(p.n_wg), dim3(kGemmWaves * kWave), lds, s, p);
    }
    return hipGetLastError();
}

template <Prec P, int RG>
static hipError_t launch_gemm_rg(GemmKind kind, int nt_qkv, const GemmParams &p, hipStream_t s, hipEvent_t e0,
                                 hipEvent_t e1) {
    switch (kind) {
    case GEMM_QKV:
        return nt_qkv == 2 ? launch_gemm_t<P, 2, RG, A_NORM, E_QKV>(p, s, e0, e1)
                           : launch_gemm_t<P, 1, RG, A_NORM, E_QKV>(p, s, e0, e1);
    case GEMM_O:
    case GEMM_DOWN:
        return launch_gemm_t<P, 1, RG, A_ACT, E_RESID>(p, s, e0, e1);
    case GEMM_GATE_UP:
        return launch_gemm_t<P, 2, RG, A_NORM, E_SWIGLU>(p, s, e0, e1);
    case GEMM_LM:
        return launch_gemm_t<P, kLmTiles, RG, A_NORM, E_ARGMAX>(p, s, e0, e1);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemm(GemmKind kind, bool bf16, int rg, int nt_qkv, const GemmParams &p, hipStream_t s,
                       hipEvent_t e0, hipEvent_t e1) {
    if (bf16) {
        if (rg == 1) return launch_gemm_rg<Prec::BF16, 1>(kind, nt_qkv, p, s, e0, e1);
        if (rg == 2) return launch_gemm_rg<Prec::BF16, 2>(kind, nt_qkv, p, s, e0, e1);
        return launch_gemm_rg<Prec::BF16, 4>(kind, nt_qkv, p, s, e0, e1);
    }
    if (rg == 1) return launch_gemm_rg<Prec::F32, 1>(kind, nt_qkv, p, s, e0, e1);
    if (rg == 2) return launch_gemm_rg<Prec::F32, 2>(kind, nt_qkv, p, s, e0, e1);
    return launch_gemm_rg<Prec::F32, 4>(kind, nt_qkv, p, s, e0, e1);
}

hipError_t launch_embed(bool bf16, int rows, const EmbedParams &p, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    auto kern = bf16 ? embed_kernel<Prec::BF16> : embed_kernel<Prec::F32>;
    if (e0)
        hipExtLaunchKernelGGL(kern, dim3(rows), dim3(256), 0, s, e0, e1, 0, p);
    else
        hipLaunchKernelGGL(kern, dim3(rows), dim3(256), 0, s, p);
    return hipGetLastError();
}

template <Prec P>
static hipError_t launch_attn_p(int rg, const AttnParams &p, int nch_launch, hipStream_t s, hipEvent_t e0,
                                hipEvent_t e1) {
    dim3 grid(nch_launch, p.n_heads);
    auto kern = rg == 1 ? attn_partial_kernel<P, 1> : (rg == 2 ? attn_partial_kernel<P, 2> : attn_partial_kernel<P, 4>);
    if (e0)
        hipExtLaunchKernelGGL(kern, grid, dim3(kWave * rg), 0, s, e0, e1, 0, p);
    else
        hipLaunchKernelGGL(kern, grid, dim3(kWave * rg), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_attn(bool bf16, int rg, int nch_launch, const AttnParams &p, hipStream_t s, hipEvent_t e0,
                       hipEvent_t e1) {
    return bf16 ? launch_attn_p<Prec::BF16>(rg, p, nch_launch, s, e0, e1)
                : launch_attn_p<Prec::F32>(rg, p, nch_launch, s, e0, e1);
}

hipError_t launch_attn_combine(bool bf16, int rows, const AttnParams &p, hipStream_t s, hipEvent_t e0,
                               hipEvent_t e1) {
    dim3 grid(p.n_heads, rows);
    auto kern = bf16 ? attn_combine_kernel<Prec::BF16> : attn_combine_kernel<Prec::F32>;
    if (e0)
        hipExtLaunchKernelGGL(kern, grid, dim3(p.hd), 0, s, e0, e1, 0, p);
    else
        hipLaunchKernelGGL(kern, grid, dim3(p.hd), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_scan(const ScanParams &p, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    if (e0)
        hipExtLaunchKernelGGL(scan_commit_kernel, dim3(1), dim3(kWave), 0, s, e0, e1, 0, p);
    else
        hipLaunchKernelGGL(scan_commit_kernel, dim3(1), dim3(kWave), 0, s, p);
    return hipGetLastError();
}

__global__ void setup_kernel(SetupParams p) {
    Ctl *c = p.ctl;
    const int i = threadIdx.x;
    if (i < p.m) c->z[i] = p.z[i];
    if (i == 0) {
        c->mode = p.mode;
        c->m = p.m;
        if (p.set_L) {
            c->L = p.L;
            c->err = 0;
            c->done = 0;
        }
    }
}

hipError_t launch_setup(const SetupParams &p, hipStream_t s) {
    hipLaunchKernelGGL(setup_kernel, dim3(1), dim3(kWave), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_decode_init(const ScanParams &p, hipStream_t s) {
    hipLaunchKernelGGL(decode_init_kernel, dim3(1), dim3(kWave), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_repack(bool bf16, const void *src, const int32_t *perm, int K, int Ks, int n_tiles, uint8_t *dst,
                         hipStream_t s) {
    const size_t tiles = (size_t)n_tiles * Ks;
    const unsigned gx = (unsigned)(tiles < 65535 ? tiles : 65535);
    const unsigned gy = (unsigned)((tiles + gx - 1) / gx);
    if (bf16)
        hipLaunchKernelGGL(repack_kernel<Prec::BF16>, dim3(gx, gy), dim3(kWave), 0, s, src, perm, K, Ks, n_tiles, dst);
    else
        hipLaunchKernelGGL(repack_kernel<Prec::F32>, dim3(gx, gy), dim3(kWave), 0, s, src, perm, K, Ks, n_tiles, dst);
    return hipGetLastError();
}

}  // namespace cllm
