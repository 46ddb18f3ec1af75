// HIP kernels of one Jacobi iteration on gfx950 (CDNA4).
//
// An iteration over a block of m tokens at positions L .. L+m-1 (Section 3.1: one causal forward
// pass over the n-token block gives all n greedy predictions) is the launch sequence
//   embed -> per layer [QKV GEMM (+RMSNorm prologue, +RoPE, +provisional KV write)
//                       -> attention partials -> attention combine
//                       -> O GEMM (+residual) -> gate/up GEMM (+RMSNorm prologue, +SwiGLU)
//                       -> down GEMM (+residual)]
//   -> LM-head GEMM (+RMSNorm prologue, +argmax partials) -> scan/commit.
// A batched iteration runs the blocks of several sequences at once (their rows packed one after
// another). Every kernel reads the rows, their sequences and positions from the device row
// table, so the same launch sequence serves every iteration without host round trips.
//
// Determinism: every reduction has a fixed order that depends only on the model shape, never on
// the number of rows or their packing, so a row's results do not depend on how many rows (or
// which other sequences) share the iteration. Hence greedy decoding with blocks of one token
// (AR), Jacobi decoding and batched Jacobi decoding produce bit-identical tokens.
#include <hip/hip_ext.h>

#include <type_traits>

#include "device.h"
#include "launch.h"

namespace cllm {

// ------------------------------------------------------------------------------------------
// Weight-streaming GEMM:  Y[rows x N] = A[rows x K] * W^T,  W packed in 1 KiB tiles.
//
// Packed layout: tile (t, s) covers weight rows 16t .. 16t+15 (after the per-GEMM row order)
// and K indices s*KSTEP .. s*KSTEP+KSTEP-1; lane l's 16 bytes are row 16t + l%16, K indices
// s*KSTEP + (l/16)*VEC .. +VEC. Tiles are stored k-step major: tile (t, s) at index s * T + t
// (T tiles per k-step), so the tiles every workgroup reads for one k-step are one contiguous
// region (measured 1-7% faster streaming than row blocks contiguous over s).
//
// A workgroup of 8 waves owns NT consecutive tiles (16*NT output columns) for all rows; wave w
// takes k-steps w, w+8, w+16, ... and accumulates them in order with MFMA; the 8 partial tiles
// are then summed in a fixed tree ((w0+w4)+(w2+w6))+((w1+w5)+(w3+w7)). Weights are read once,
// straight into registers (no LDS); the activation rows (a few KiB, L2-resident) are re-read.
// In bf16 the activations are fp32 values split into hi and lo bf16 planes, and each k-step runs
// one MFMA per plane against the same weight tile: products are exact in fp32, so the operand
// keeps 16 significant bits instead of bf16's 8.
//
// Products that follow an RMSNorm take the operand x (.) g written by the producer of x and
// scale each output row by 1/sqrt(mean(x^2) + eps), reduced from the producer's per-16-column
// sums of squares.
// ------------------------------------------------------------------------------------------

enum Epi { E_QKV = 0, E_RESID = 1, E_SWIGLU = 2, E_ARGMAX = 3, E_LOGITS = 4 };

template <Prec P, int NT, int RG>
struct Stage {  // operands of one k-step
    u32x4 b[NT];                      // weight tiles
    u32x4 a[PrecT<P>::PLANES][RG];    // activation rows (hi, lo planes for bf16)
};

// Loads of one k-step s (callers clamp s into [0, Ks), so every load is issued and the compiler
// can count outstanding loads exactly). Tiles past the last one (a ragged last workgroup) load
// the last tile again; their columns are never written. SHARED: the weight tiles are read by
// several workgroups (the row tiles of one column group), so they are loaded as ordinary
// (cached) loads; otherwise they are streamed (nontemporal: read once, not kept in the caches).
template <Prec P, int NT, int RG, bool SHARED>
__device__ __forceinline__ void gemm_load(Stage<P, NT, RG> &st, const GemmParams &p, int t0, int rg0, int s, int lane) {
    using PT = PrecT<P>;
    using T = typename PT::T;
    const int tiles = p.cols >> 4;
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const u32x4 *src =
            reinterpret_cast<const u32x4 *>(p.W + ((size_t)s * tiles + min(t0 + j, tiles - 1)) * kTileBytes) + lane;
        st.b[j] = SHARED ? *src : __builtin_nontemporal_load(src);
    }
    const T *A = reinterpret_cast<const T *>(p.A);
    const int ks_a = p.lda / PT::KSTEP;
#pragma unroll
    for (int pl = 0; pl < PT::PLANES; ++pl)
#pragma unroll
        for (int r = 0; r < RG; ++r)
            st.a[pl][r] = *reinterpret_cast<const u32x4 *>(A + pl * act_plane(p.rr.cap, p.lda) +
                                                          ((size_t)((rg0 + r) * ks_a + s) * kWave + lane) * PT::VEC);
}

// MFMAs of one k-step: every hi-plane product, then every lo-plane product (bf16).
template <Prec P, int NT, int RG>
__device__ __forceinline__ void gemm_compute(const Stage<P, NT, RG> &st, f32x4 (&acc)[RG][NT]) {
#pragma unroll
    for (int pl = 0; pl < PrecT<P>::PLANES; ++pl)
#pragma unroll
        for (int r = 0; r < RG; ++r)
#pragma unroll
            for (int j = 0; j < NT; ++j) acc[r][j] = mfma_kstep<P>(st.a[pl][r], st.b[j], acc[r][j]);
}

__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

// Row factor 1/sqrt(mean(x^2) + eps) of the rows [row0, row0 + ROWS) from the producer's
// per-16-column sums of squares (layout [row][T], T a multiple of 4). 32 threads per row each add
// a contiguous run of q = 4 * ceil(T/128) partials in order (16-byte reads), then a fixed xor tree
// over the row's 32 threads; the scheme depends only on T, never on the number of rows. The
// first two vectors of the first row pass are requested early by row_factor_preload. The caller's
// next barrier publishes s_inv.
template <int W>
__device__ __forceinline__ void row_factor_preload(const GemmParams &p, int row0, int tid, f32x4 (&sq_pre)[2]) {
    const int sq_part = tid & 31, sq_q = ((p.T + 127) >> 7) << 2;
    const float *src = p.ssq + (size_t)(row0 + (tid >> 5)) * p.T;
#pragma unroll
    for (int i = 0; i < 2; ++i)  // clamped, unconditional
        sq_pre[i] = *reinterpret_cast<const f32x4 *>(src + min(sq_part * sq_q + 4 * i, p.T - 4));
}

template <int W, int ROWS>
__device__ __forceinline__ void row_factor_reduce(const GemmParams &p, int row0, int tid, const f32x4 (&sq_pre)[2],
                                                  float *s_inv) {
    constexpr int RPP = W * kWave / 32;  // rows per pass
    static_assert(ROWS % RPP == 0, "row passes cover the row groups");
    const int sq_part = tid & 31, sq_q = ((p.T + 127) >> 7) << 2;
    for (int pass = 0; pass < ROWS / RPP; ++pass) {
        const int row = pass * RPP + (tid >> 5);
        const float *src = p.ssq + (size_t)(row0 + row) * p.T;
        float sum = 0.0f;
        for (int i0 = 0; i0 < sq_q; i0 += 8) {
            f32x4 v[2];
            if (pass == 0 && i0 == 0) {
                v[0] = sq_pre[0];
                v[1] = sq_pre[1];
            } else {
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    v[i] = *reinterpret_cast<const f32x4 *>(src + min(sq_part * sq_q + i0 + 4 * i, p.T - 4));
            }
#pragma unroll
            for (int i = 0; i < 8; ++i)
                if (i0 + i < sq_q && sq_part * sq_q + i0 + i < p.T) sum += v[i >> 2][i & 3];
        }
#pragma unroll
        for (int off = 16; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, 32);
        if (sq_part == 0) s_inv[row] = 1.0f / sqrtf(sum / (float)p.K + p.eps);
    }
}

// Epilogues of a finished ROWS x COLS output tile in s_tile (row stride COLS + 1) for rows
// [row0, row0 + ROWS) of the iteration (m of them live) and column workgroup wg of width COLS
// (columns at or past p.cols, in a ragged last workgroup, are dropped); s_red is scratch of at
// least ROWS x COLS floats.
template <Prec P, int NT, int RG, int EP, int W>
__device__ __forceinline__ void gemm_epilogue(const GemmParams &p, float *s_tile, float *s_red, int row0, int m, int wg,
                                              int tid, int lane, int w) {
    using T = typename PrecT<P>::T;
    constexpr int ROWS = 16 * RG, COLS = 16 * NT;
    const int t0 = wg * NT;
    if constexpr (EP == E_QKV) {
        // Packed columns -> (section, head, dim). Tile b of a head holds dims [8b, 8b+8) and
        // their rotate-half partners [hd/2+8b, hd/2+8b+8): column o of the tile and column o ^ 8
        // are partners, so every tile is complete for RoPE and a workgroup may own any number
        // of tiles.
        const int hd = p.hd, d = p.d, h2 = hd >> 1;
        for (int idx = tid; idx < ROWS * COLS; idx += W * kWave) {
            const int row = idx / COLS, pc = idx % COLS;
            const int R = t0 * 16 + pc;  // packed row index
            if (row >= m || R >= p.cols) continue;
            const int sec = R / d, within = R % d, head = within / hd;
            const int q = within % hd, b = q >> 4, o = q & 15;
            const int dim = o < 8 ? 8 * b + o : h2 + 8 * b + (o - 8);
            const int partner = pc ^ 8;
            const RowInfo ri = p.rr.rows[row0 + row];
            const int pos = ri.pos;
            const size_t kvo = (size_t)p.rr.tab->seq[ri.b] * p.kv_seq;  // this row's sequence slot
            float x = s_tile[row * (COLS + 1) + pc];
            if (sec < 2) {
                const float y = s_tile[row * (COLS + 1) + partner];
                const int j = dim < h2 ? dim : dim - h2;
                const float c = p.rcos[(size_t)pos * h2 + j], s = p.rsin[(size_t)pos * h2 + j];
                x = dim < h2 ? (x * c - y * s) : (x * c + y * s);
            }
            const T e = to_elem<P>(x);  // cached keys and values are rounded to the cache dtype
            if (sec == 0)
                put_act<P>(reinterpret_cast<T *>(p.Q), act_plane(p.rr.cap, d), act_idx<P>(row0 + row, head * hd + dim, d), x);
            else if (sec == 1)
                reinterpret_cast<T *>(p.Kc)[kvo + (size_t)head * p.ctx_alloc * hd + kcache_idx<P>(pos, dim, hd)] = e;
            else
                reinterpret_cast<T *>(p.Vt)[kvo + (size_t)head * p.ctx_alloc * hd + vcache_idx<P>(pos, dim, hd)] = e;
        }
    } else if constexpr (EP == E_RESID) {
        // X += Y over this workgroup's columns, then the per-16-column sums of squares of the
        // new rows (summed in column order) for the next RMSNorm.
        const int c0 = t0 * 16;
        float *s_sq = s_red;  // ROWS x COLS
        for (int idx = tid; idx < ROWS * COLS; idx += W * kWave) {
            const int row = idx / COLS, c = idx % COLS;
            float v = 0.0f;
            if (row < m && c0 + c < p.cols) {
                float *xp = p.Xout + (size_t)(row0 + row) * p.ldx + c0 + c;
                v = *xp + s_tile[row * (COLS + 1) + c];
                *xp = v;
                // operand of the next RMSNorm-ed product: x (.) g
                put_act<P>(reinterpret_cast<T *>(p.An), act_plane(p.rr.cap, p.ldx),
                           act_idx<P>(row0 + row, c0 + c, p.ldx), v * p.gain[c0 + c]);
            }
            s_sq[idx] = v * v;
        }
        __syncthreads();
        if (tid < ROWS * NT) {
            const int row = tid / NT, j = tid % NT;
            if (row < m && (t0 + j) * 16 < p.cols) {
                float sum = 0.0f;
#pragma unroll
                for (int c = 0; c < 16; ++c) sum += s_sq[row * COLS + 16 * j + c];
                p.ssq_out[(size_t)(row0 + row) * p.T + t0 + j] = sum;
            }
        }
    } else if constexpr (EP == E_SWIGLU) {
        // Tiles come in (gate, up) pairs of the same 16 features.
        static_assert(NT % 2 == 0, "gate/up epilogue pairs a gate tile with an up tile");
        for (int idx = tid; idx < ROWS * COLS / 2; idx += W * kWave) {
            const int row = idx / (COLS / 2), f = idx % (COLS / 2), q = f >> 4, c = f & 15;
            if (row >= m || wg * COLS + 32 * q >= p.cols) continue;  // pair past the last column
            const float gt = s_tile[row * (COLS + 1) + 32 * q + c];
            const float up = s_tile[row * (COLS + 1) + 32 * q + 16 + c];
            put_act<P>(reinterpret_cast<T *>(p.H), act_plane(p.rr.cap, p.Fp),
                       act_idx<P>(row0 + row, wg * (COLS / 2) + f, p.Fp), silu(gt) * up);
        }
    } else if constexpr (EP == E_LOGITS) {
        // Plain fp32 output rows (the loss head's logits): Zout[row][col], col < V.
        const int c0 = t0 * 16;
        for (int idx = tid; idx < ROWS * COLS; idx += W * kWave) {
            const int row = idx / COLS, c = idx % COLS;
            if (row < m && c0 + c < p.V) p.Zout[(size_t)(row0 + row) * p.ldz + c0 + c] = s_tile[row * (COLS + 1) + c];
        }
    } else {  // E_ARGMAX
        // One wave per row: (max, lowest column) over this workgroup's columns < V.
        for (int row = w; row < ROWS; row += W) {
            if (row >= m) break;
            float bv = -INFINITY;
            int bi = 0x7fffffff;
            int nan = 0;
            for (int c = lane; c < COLS; c += kWave) {
                const int col = t0 * 16 + c;
                if (col < p.V) {
                    const float v = s_tile[row * (COLS + 1) + c];
                    if (p.dbg) p.dbg[(size_t)(row0 + row) * p.V + col] = v;
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
                p.pmax[(size_t)wg * p.rr.cap + row0 + row] = bv;
                p.pidx[(size_t)wg * p.rr.cap + row0 + row] = nan ? -1 : bi;
            }
        }
    }
}

template <Prec P, int NT, int RG, int EP, int D, int W, bool MT>
__global__ __launch_bounds__(W * kWave) void gemm_kernel(GemmParams p) {
    static_assert(W == 8, "the K split and its reduction tree are defined for 8 waves");
    constexpr bool ROWSCALE = EP != E_RESID && EP != E_LOGITS;  // the product follows an RMSNorm
    constexpr int ROWS = 16 * RG, COLS = 16 * NT;
    const int wg = blockIdx.x;  // column group
    if constexpr (EP == E_LOGITS) {
        if (p.kc > 0) {  // split K: k-steps [z kc, min((z + 1) kc, Ks)), partial products to plane z
            const int ks0 = blockIdx.z * p.kc;
            p.W += (size_t)ks0 * (p.cols >> 4) * kTileBytes;
            p.A = reinterpret_cast<const uint8_t *>(p.A) + (size_t)ks0 * kWave * 16;  // 16-byte lane vectors
            p.Ks = min(p.kc, p.Ks - ks0);
            p.Zout += (size_t)blockIdx.z * p.zstride;
        }
    }
    // This workgroup's row tile: rows [row0, row0 + ROWS) of the iteration (within the row
    // capacity); m of them are live. A launch of one row tile (MT false) always has live rows, so
    // nothing waits for the row count before the first loads; with several row tiles (MT) a tile
    // with no live row exits first.
    const int row0 = (p.rt0 + (int)blockIdx.y) * ROWS;
    request_together(p.W, p.A, p.ssq, p.Ks, p.cols, p.lda, p.rr.cap, p.T);
    const int m = p.rr.tab->R - row0;
    if constexpr (MT) {
        if (m <= 0) return;
    }
    const int rg0 = row0 >> 4;
    const int tid = threadIdx.x, lane = tid & 63;
    // wave index made explicitly wave-uniform, so k-step addresses live in scalar registers and
    // every load shares one per-lane offset
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int t0 = wg * NT;

    extern __shared__ float smem[];
    float *s_red = smem;                   // W waves x NT x 256 (also ROWS x COLS for E_RESID)
    float *s_tile = s_red + W * NT * 256;  // ROWS x (COLS + 1)
    float *s_inv = s_tile + ROWS * (COLS + 1);      // ROWS

    // Row factor inputs are requested before the weights (their latency overlaps the first
    // k-step's) and reduced after the main loop.
    f32x4 sq_pre[2];
    if constexpr (ROWSCALE) row_factor_preload<W>(p, row0, tid, sq_pre);

    // This wave's k-steps (nmy of them); the first D-1 are requested first.
    const int nmy = w < p.Ks ? (p.Ks - w + W - 1) / W : 0;
    auto step_of = [&](int q) { return min(w + q * W, p.Ks - 1); };
    Stage<P, NT, RG> ring[D];
#pragma unroll
    for (int j = 0; j < D - 1; ++j) gemm_load<P, NT, RG, MT>(ring[j], p, t0, rg0, step_of(j), lane);

    f32x4 acc[RG][NT];
#pragma unroll
    for (int r = 0; r < RG; ++r)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[r][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Software pipeline: a ring of D k-steps whose loads are in flight while the oldest one's
    // MFMAs run. The steady state is branch-free (exact wait counts); the drain issues no loads
    // past the end.
    if (nmy > 0) {
        // blocks of D steps whose prefetches (up to step b*D + 2D - 2) are all in range
        const int nfull = nmy >= 2 * D - 1 ? (nmy - (D - 1)) / D : 0;
        for (int bi = 0; bi < nfull; ++bi) {
#pragma unroll
            for (int j = 0; j < D; ++j) {
                // sched_barrier keeps the scheduler from sinking loads to their uses.
                gemm_load<P, NT, RG, MT>(ring[(j + D - 1) % D], p, t0, rg0, step_of(bi * D + j + D - 1), lane);
                __builtin_amdgcn_sched_barrier(0);
                gemm_compute(ring[j], acc);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        const int v0 = nfull * D;
#pragma unroll
        for (int j = 0; j < 2 * D - 1; ++j) {
            const int v = v0 + j;
            if (v < nmy) {
                if (v + D - 1 < nmy)
                    gemm_load<P, NT, RG, MT>(ring[(j + D - 1) % D], p, t0, rg0, step_of(v + D - 1), lane);
                gemm_compute(ring[j % D], acc);
            }
        }
    }

    if constexpr (ROWSCALE) row_factor_reduce<W, ROWS>(p, row0, tid, sq_pre, s_inv);

    // Sum of the 8 waves' partial tiles through LDS, one row group at a time, in the fixed tree
    // ((w0+w4)+(w2+w6))+((w1+w5)+(w3+w7)); then the RMSNorm row factor.
#pragma unroll
    for (int r = 0; r < RG; ++r) {
#pragma unroll
        for (int j = 0; j < NT; ++j)
            *reinterpret_cast<f32x4 *>(s_red + ((size_t)(w * NT + j) * 64 + lane) * 4) = acc[r][j];
        __syncthreads();
        for (int e = tid; e < NT * 256; e += W * kWave) {
            float x[W];
#pragma unroll
            for (int q = 0; q < W; ++q) x[q] = s_red[(size_t)q * NT * 256 + e];
            float sum = ((x[0] + x[4]) + (x[2] + x[6])) + ((x[1] + x[5]) + (x[3] + x[7]));
            // element e = (tile j, lane l, register v); C layout: row 4*(l/16)+v, column l%16
            const int j = e >> 8, l = (e >> 2) & 63, v = e & 3;
            const int row = 16 * r + 4 * (l >> 4) + v;
            if constexpr (ROWSCALE) sum *= s_inv[row];
            s_tile[row * (COLS + 1) + 16 * j + (l & 15)] = sum;
        }
        __syncthreads();
    }

    gemm_epilogue<P, NT, RG, EP, W>(p, s_tile, s_red, row0, m, wg, tid, lane, w);
}

// ------------------------------------------------------------------------------------------
// Embedding gather: X[i] = E[z_i] (fp32), the operand X[i] (.) g of the first layer's QKV product
// and the per-16-column sums of squares for its RMSNorm.
// ------------------------------------------------------------------------------------------
template <Prec P>
__global__ __launch_bounds__(256) void embed_kernel(EmbedParams p) {
    using PT = PrecT<P>;
    using T = typename PT::T;
    constexpr int V16 = 16 / sizeof(T);  // elements per 16-byte vector
    static_assert(V16 == PT::VEC, "an operand vector is one 16-byte load");
    const int row = blockIdx.x;  // < row capacity (launcher)
    request_together(p.rr.tab, p.rr.rows, p.rr.cap, p.E, p.X, p.ssq, p.An, p.gain, p.d);
    const int R = p.rr.tab->R, tok = p.rr.rows[row].tok;
    request_together(R, tok);
    if (row >= R) return;
    const T *e = reinterpret_cast<const T *>(p.E) + (size_t)tok * p.d;
    float *x = p.X + (size_t)row * p.d;
    T *an = reinterpret_cast<T *>(p.An);
    for (int t = threadIdx.x; t < p.d / 16; t += blockDim.x) {  // one 16-column tile per thread
        alignas(16) T ev[16];
        alignas(16) T av[PT::PLANES][16];
        alignas(16) float xv[16];
        alignas(16) float gv[16];
#pragma unroll
        for (int q = 0; q < 16 / V16; ++q)
            *reinterpret_cast<u32x4 *>(ev + q * V16) = *reinterpret_cast<const u32x4 *>(e + 16 * t + q * V16);
#pragma unroll
        for (int q = 0; q < 4; ++q)
            *reinterpret_cast<f32x4 *>(gv + 4 * q) = *reinterpret_cast<const f32x4 *>(p.gain + 16 * t + 4 * q);
        float sum = 0.0f;
#pragma unroll
        for (int c = 0; c < 16; ++c) {
            xv[c] = from_elem<P>(ev[c]);
            const float a = xv[c] * gv[c];
            av[0][c] = to_elem<P>(a);
            if constexpr (PT::PLANES == 2) av[PT::PLANES - 1][c] = to_elem<P>(a - from_elem<P>(av[0][c]));
            sum += xv[c] * xv[c];
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) *reinterpret_cast<f32x4 *>(x + 16 * t + 4 * q) = *reinterpret_cast<f32x4 *>(xv + 4 * q);
#pragma unroll
        for (int pl = 0; pl < PT::PLANES; ++pl)
#pragma unroll
            for (int q = 0; q < 16 / V16; ++q)  // V16 == VEC: one vector is contiguous in the packed layout
                *reinterpret_cast<u32x4 *>(an + pl * act_plane(p.rr.cap, p.d) + act_idx<P>(row, 16 * t + q * V16, p.d)) =
                    *reinterpret_cast<u32x4 *>(&av[pl][q * V16]);
        p.ssq[(size_t)row * (p.d / 16) + t] = sum;
    }
}

// ------------------------------------------------------------------------------------------
// Block-causal attention in one kernel, for launches whose rows see at most kFusedChunks
// chunks. Workgroup (16-dim output slice dt, head h; 16-row group of a batch entry), 8 waves:
// wave w computes chunks w, w+8, ... exactly as attn_partial_kernel computes them (chunk max,
// sum and unnormalised output of this slice, per row) into LDS; the workgroup then combines the
// chunks up to each row's position exactly as attn_combine_kernel does (same weights, same
// chunk order). Every value is therefore bit-identical to the two-kernel path, whichever of the
// two a launch takes. Each workgroup of a head reads the head's whole K and one 16-dim slice of
// V; the slices of a head are dispatched to one XCD (block index dt * n_heads + h with n_heads
// a multiple of 8), so its L2 serves the K re-reads.
// ------------------------------------------------------------------------------------------
constexpr int kAttnWaves = 8;

template <Prec P, int HD>
struct AttnChunk {  // one chunk's operands in registers
    u32x4 k[4][HD / PrecT<P>::KSTEP];
    u32x4 v[4];  // bf16: v[0..1] (keys 32kp..); fp32: v[0..3] (keys 16kt..)
};

template <Prec P, int HD>
__device__ __forceinline__ void attn_load_chunk(AttnChunk<P, HD> &ch, const typename PrecT<P>::T *Kh,
                                                const typename PrecT<P>::T *Vh, int c, int dt, int lane) {
    using PT = PrecT<P>;
    constexpr int NKK = HD / PT::KSTEP, NDT = HD / 16;
    const int key0 = c * kAttnChunk;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
            ch.k[kt][kk] = *reinterpret_cast<const u32x4 *>(Kh + ((size_t)((key0 >> 4) + kt) * NKK + kk) * (kWave * PT::VEC) +
                                                            lane * PT::VEC);
    if constexpr (P == Prec::BF16) {
#pragma unroll
        for (int kp = 0; kp < 2; ++kp)
            ch.v[kp] = *reinterpret_cast<const u32x4 *>(Vh + ((size_t)((key0 >> 5) + kp) * NDT + dt) * (kWave * 8) + lane * 8);
    } else {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
            ch.v[kt] = *reinterpret_cast<const u32x4 *>(Vh + ((size_t)((key0 >> 4) + kt) * NDT + dt) * (kWave * 4) + lane * 4);
    }
}

template <Prec P, int HD>
__global__ __launch_bounds__(kAttnWaves * kWave) void attn_kernel(AttnParams p) {
    using PT = PrecT<P>;
    using T = typename PT::T;
    constexpr int NKK = HD / PT::KSTEP;
    constexpr int W = kAttnWaves;
    const RowTab *tab = p.rr.tab;
    request_together(tab, p.Q, p.Kc, p.Vt, p.kv_seq, p.ctx_alloc, p.rr.cap, p.d, p.n_heads);
    const int h = blockIdx.x % p.n_heads, dt = blockIdx.x / p.n_heads;
    const int rgi = blockIdx.y, b = blockIdx.z;  // b < kMaxSeqs (launcher)
    const int nseq = tab->nseq, m = tab->m[b], L = tab->L[b], r0 = tab->r0[b], slot = tab->seq[b];
    request_together(nseq, m, L, r0, slot);
    if (b >= nseq || 16 * rgi >= m) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, r16 = lane & 15;
    const int d = p.d;
    const int qi = 16 * rgi + r16;              // row within the block
    const int qld = min(r0 + qi, p.rr.cap - 1);  // rows past the block load in-bounds filler
    const int qpos = L + qi;
    // chunks holding a key visible to some row of the group (<= kFusedChunks: the launcher's bound)
    const int nvis = min((L + min(m - 1, 16 * rgi + 15)) / kAttnChunk + 1, kFusedChunks);
    const size_t kvo = (size_t)slot * p.kv_seq + (size_t)h * p.ctx_alloc * HD;
    const T *Kh = reinterpret_cast<const T *>(p.Kc) + kvo;
    const T *Vh = reinterpret_cast<const T *>(p.Vt) + kvo;
    const T *Q = reinterpret_cast<const T *>(p.Q);

    // per chunk and row: max, sum, and the slice's 16 unnormalised output dims
    __shared__ float s_mc[kFusedChunks][16], s_lc[kFusedChunks][16], s_oc[kFusedChunks][16][17];

    // This wave's chunks w, w + W, ... (nmine of them); the loads of the next one are in flight
    // while a chunk is computed (the index is clamped, so the last prefetch stays in bounds).
    const int nmine = w < nvis ? (nvis - 1 - w) / W + 1 : 0;
    auto chunk_of = [&](int i) { return min(w + i * W, nvis - 1); };
    u32x4 qv[PT::PLANES][NKK];
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
        for (int pl = 0; pl < PT::PLANES; ++pl)
            qv[pl][kk] = *reinterpret_cast<const u32x4 *>(
                Q + pl * act_plane(p.rr.cap, d) + act_idx<P>(qld, h * HD + kk * PT::KSTEP + g * PT::VEC, d));
    AttnChunk<P, HD> buf[2];
    attn_load_chunk<P, HD>(buf[0], Kh, Vh, chunk_of(0), dt, lane);

    auto process = [&](const AttnChunk<P, HD> &ch, int c) {
        const int key0 = c * kAttnChunk;
        f32x4 st[4];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
            st[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int pl = 0; pl < PT::PLANES; ++pl)
#pragma unroll
                for (int kk = 0; kk < NKK; ++kk) st[kt] = mfma_kstep<P>(ch.k[kt][kk], qv[pl][kk], st[kt]);
        }
        // st[kt][v] = S^T[key0 + 16kt + 4g + v][row r16]
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int key = key0 + 16 * kt + 4 * g + v;
                const float sc = key <= qpos ? st[kt][v] * p.scale_log2 : -INFINITY;
                st[kt][v] = sc;
                mx = fmaxf(mx, sc);
            }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        float l = 0.0f;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const float pr = (mx == -INFINITY || st[kt][v] == -INFINITY) ? 0.0f : exp2f(st[kt][v] - mx);
                st[kt][v] = pr;
                l += pr;
            }
        l += __shfl_xor(l, 16);
        l += __shfl_xor(l, 32);
        f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
        if constexpr (P == Prec::BF16) {
#pragma unroll
            for (int kp = 0; kp < 2; ++kp) {
                // P = hi + lo, hi = bf16(P), lo = bf16(P - hi): the probabilities keep ~2^-17
                const f32x4 pa = st[2 * kp], pb = st[2 * kp + 1];
                const float pv[8] = {pa[0], pa[1], pa[2], pa[3], pb[0], pb[1], pb[2], pb[3]};
                uint32_t hi[8], lo[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    hi[q] = f2bf(pv[q]);
                    lo[q] = f2bf(pv[q] - bf2f((uint16_t)hi[q]));
                }
                const u32x4 bhi = u32x4{hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16), hi[4] | (hi[5] << 16),
                                        hi[6] | (hi[7] << 16)};
                const u32x4 blo = u32x4{lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16), lo[4] | (lo[5] << 16),
                                        lo[6] | (lo[7] << 16)};
                o = mfma_kstep<P>(ch.v[kp], bhi, o);
                o = mfma_kstep<P>(ch.v[kp], blo, o);
            }
        } else {
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) {
                const f32x4 pk = st[kt];
                o = mfma_kstep<P>(ch.v[kt], u32x4{__float_as_uint(pk[0]), __float_as_uint(pk[1]), __float_as_uint(pk[2]),
                                                  __float_as_uint(pk[3])},
                                  o);
            }
        }
        // o[v] = O^T[16dt + 4g + v][row r16]
        if (g == 0) {
            s_mc[c][r16] = mx;
            s_lc[c][r16] = l;
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) s_oc[c][r16][4 * g + v] = o[v];
    };
    for (int i = 0; i < nmine; i += 2) {
        attn_load_chunk<P, HD>(buf[1], Kh, Vh, chunk_of(i + 1), dt, lane);
        process(buf[0], w + i * W);
        if (i + 1 >= nmine) break;
        attn_load_chunk<P, HD>(buf[0], Kh, Vh, chunk_of(i + 2), dt, lane);
        process(buf[1], w + (i + 1) * W);
    }
    __syncthreads();

    // Combine the chunks up to the row's own position in chunk order (as attn_combine_kernel).
    if (tid < 256) {
        const int row = tid >> 4, dim = tid & 15;
        if (16 * rgi + row < m) {
            const int nlive = min((L + 16 * rgi + row) / kAttnChunk + 1, nvis);
            float M = -INFINITY;
            for (int c = 0; c < nlive; ++c) M = fmaxf(M, s_mc[c][row]);
            float num = 0.0f, den = 0.0f;
            for (int c = 0; c < nlive; ++c) {
                const float mc = s_mc[c][row];
                const float wc = mc == -INFINITY ? 0.0f : exp2f(mc - M);
                den += wc * s_lc[c][row];
                num += wc * s_oc[c][row][dim];
            }
            put_act<P>(reinterpret_cast<T *>(p.O), act_plane(p.rr.cap, d),
                       act_idx<P>(r0 + 16 * rgi + row, h * HD + 16 * dt + dim, d), num / den);
        }
    }
}

// ------------------------------------------------------------------------------------------
// Block-causal attention, split over fixed 64-key chunks at absolute positions.
// Workgroup (chunk c, head h), one wave per 16 query rows. With the cache K [pos][d] and the
// transposed value cache Vt [d][pos]:
//   S^T = K_chunk * Q^T   (MFMA A operand = key rows, B operand = query rows; bf16 queries as
//                          hi and lo planes, one MFMA each)
//   softmax over keys j <= L + i (fp32, base-2 exponent with the 1/sqrt(hd) scale folded in)
//   O^T = Vt_chunk * P^T  (the lane's own S^T registers are the B operand; the V^T loads use
//                          the same K-slot assignment)
// Each (h, c, row) writes a partial (max, sum, unnormalised output).
// ------------------------------------------------------------------------------------------
template <Prec P, int HD, int RG>
__global__ __launch_bounds__(kWave * RG) void attn_partial_kernel(AttnParams p) {
    using PT = PrecT<P>;
    using T = typename PT::T;
    constexpr int NKK = HD / PT::KSTEP;  // k-steps of the score product
    constexpr int NDT = HD / 16;         // 16-dim tiles of the output
    const RowTab *tab = p.rr.tab;
    request_together(tab, p.nrb, p.Q, p.Kc, p.Vt, p.kv_seq, p.ctx_alloc, p.rr.cap, p.d, p.nch);
    const int b = blockIdx.z / p.nrb;            // batch entry (< kMaxSeqs: the launcher checks)
    const int rbase = (blockIdx.z % p.nrb) * 16 * RG;  // first block row of this workgroup
    // the entry's fields are requested together, before any of them is tested
    const int nseq = tab->nseq, m = tab->m[b], L = tab->L[b], r0 = tab->r0[b], slot = tab->seq[b];
    request_together(nseq, m, L, r0, slot);
    if (b >= nseq) return;
    if (rbase >= m) return;
    const int c = blockIdx.x, h = blockIdx.y;
    const int key0 = c * kAttnChunk;
    if (key0 > L + min(m - 1, rbase + 16 * RG - 1)) return;  // no key of this chunk is visible to any row
    const int lane = threadIdx.x & 63, rg = threadIdx.x >> 6;
    if (rbase + 16 * rg >= m) return;  // this wave's rows are all past the block
    const int g = lane >> 4, r16 = lane & 15;
    const int d = p.d;
    const int qi = rbase + 16 * rg + r16;   // row within the block
    const int qrow = r0 + qi;               // row of the iteration
    const int qld = min(qrow, p.rr.cap - 1);  // rows past the block load in-bounds filler
    const int qpos = L + qi;
    // this head's caches of this sequence slot (operand order: one contiguous KiB per load)
    const size_t kvo = (size_t)slot * p.kv_seq + (size_t)h * p.ctx_alloc * HD;
    const T *Kh = reinterpret_cast<const T *>(p.Kc) + kvo;
    const T *Vh = reinterpret_cast<const T *>(p.Vt) + kvo;
    const T *Q = reinterpret_cast<const T *>(p.Q);

    // Every load of the workgroup is issued up front: Q rows, the chunk's 64 keys and values.
    u32x4 qv[PT::PLANES][NKK], kv[4][NKK];
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
        const int dcol = h * HD + kk * PT::KSTEP + g * PT::VEC;
#pragma unroll
        for (int pl = 0; pl < PT::PLANES; ++pl)
            qv[pl][kk] = *reinterpret_cast<const u32x4 *>(Q + pl * act_plane(p.rr.cap, d) + act_idx<P>(qld, dcol, d));
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)  // keys key0 + 16kt + lane%16, dims kk*KSTEP + (lane/16)*VEC ..
            kv[kt][kk] = *reinterpret_cast<const u32x4 *>(
                Kh + ((size_t)((key0 >> 4) + kt) * NKK + kk) * (kWave * PT::VEC) + lane * PT::VEC);
    }
    // V^T operand: row = dim 16*dt + lane%16; K slots = keys 32kp+4g+(0..3), 32kp+16+4g+(0..3) (bf16),
    // or keys 16kt+4g+(0..3) (fp32); the cache holds exactly these 16 bytes per lane contiguously.
    u32x4 vv[NDT][2];
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
        if constexpr (P == Prec::BF16) {
#pragma unroll
            for (int kp = 0; kp < 2; ++kp)
                vv[dt][kp] = *reinterpret_cast<const u32x4 *>(
                    Vh + ((size_t)((key0 >> 5) + kp) * NDT + dt) * (kWave * 8) + lane * 8);
        }
    }

    f32x4 st[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
        st[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int pl = 0; pl < PT::PLANES; ++pl)
#pragma unroll
            for (int kk = 0; kk < NKK; ++kk) st[kt] = mfma_kstep<P>(kv[kt][kk], qv[pl][kk], st[kt]);
    }
    // st[kt][v] = S^T[key0 + 16kt + 4g + v][qrow]
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int key = key0 + 16 * kt + 4 * g + v;
            const float sc = key <= qpos ? st[kt][v] * p.scale_log2 : -INFINITY;
            st[kt][v] = sc;
            mx = fmaxf(mx, sc);
        }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    float l = 0.0f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float pr = (mx == -INFINITY || st[kt][v] == -INFINITY) ? 0.0f : exp2f(st[kt][v] - mx);
            st[kt][v] = pr;
            l += pr;
        }
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);

    const bool live = qi < m;  // rows past the block belong to the next entry: not written
    const size_t pbase = ((size_t)h * p.nch + c) * p.rr.cap + qrow;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
        f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
        if constexpr (P == Prec::BF16) {
#pragma unroll
            for (int kp = 0; kp < 2; ++kp) {
                // P = hi + lo with hi = bf16(P), lo = bf16(P - hi): two bf16 products carry P to
                // ~2^-17 relative, so the probabilities are not rounded to bf16.
                const f32x4 pa = st[2 * kp], pb = st[2 * kp + 1];
                const float pv[8] = {pa[0], pa[1], pa[2], pa[3], pb[0], pb[1], pb[2], pb[3]};
                uint32_t hi[8], lo[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    hi[q] = f2bf(pv[q]);
                    lo[q] = f2bf(pv[q] - bf2f((uint16_t)hi[q]));
                }
                const u32x4 bhi = u32x4{hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16), hi[4] | (hi[5] << 16),
                                        hi[6] | (hi[7] << 16)};
                const u32x4 blo = u32x4{lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16), lo[4] | (lo[5] << 16),
                                        lo[6] | (lo[7] << 16)};
                o = mfma_kstep<P>(vv[dt][kp], bhi, o);
                o = mfma_kstep<P>(vv[dt][kp], blo, o);
            }
        } else {
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) {
                const u32x4 va = *reinterpret_cast<const u32x4 *>(
                    Vh + ((size_t)((key0 >> 4) + kt) * NDT + dt) * (kWave * 4) + lane * 4);
                const f32x4 pk = st[kt];
                o = mfma_kstep<P>(va, u32x4{__float_as_uint(pk[0]), __float_as_uint(pk[1]), __float_as_uint(pk[2]),
                                            __float_as_uint(pk[3])},
                                  o);
            }
        }
        // o[v] = O^T[16dt + 4g + v][qrow]
        if (live) *reinterpret_cast<f32x4 *>(p.Opart + pbase * HD + 16 * dt + 4 * g) = o;
    }
    if (g == 0 && live) {
        p.Mpart[pbase] = mx;
        p.Lpart[pbase] = l;
    }
}

// Combine the chunk partials of one (head, row) in chunk order and write the O operand.
// Wave 0 derives the chunk weights w_c = 2^(m_c - M) into LDS; every thread (one output dim)
// then sums w_c * O_c in chunk order. The loads are issued in two rounds: the row count and the
// row's position, then the chunk maxima, sums and the first kCombinePre chunks' values together.
constexpr int kCombinePre = 16;  // chunks whose values are requested with the maxima

template <Prec P>
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnParams p) {
    using T = typename PrecT<P>::T;
    const int h = blockIdx.x, row = blockIdx.y;  // row < row capacity (launcher)
    request_together(p.rr.tab, p.rr.rows, p.rr.cap, p.Mpart, p.Lpart, p.Opart, p.nch, p.hd);
    const int R = p.rr.tab->R;
    const int pos = p.rr.rows[row].pos;
    request_together(R, pos);
    if (row >= R) return;
    // chunks holding a key at or before this row's position (later chunks hold none)
    const int nlive = pos / kAttnChunk + 1;
    const int tid = threadIdx.x;
    const int cap = p.rr.cap;
    const size_t b0 = (size_t)h * p.nch * cap + row;
    __shared__ float s_w[kMaxChunks], s_l[kMaxChunks];
    __shared__ float s_den;
    const int dim = tid;
    const bool has_dim = dim < p.hd;
    float pre[kCombinePre];
#pragma unroll
    for (int c = 0; c < kCombinePre; ++c)
        pre[c] = (has_dim && c < nlive) ? p.Opart[(b0 + (size_t)c * cap) * p.hd + dim] : 0.0f;
    if (tid < kWave) {
        float M = -INFINITY;
        for (int c = tid; c < nlive; c += kWave) {
            const float mc = p.Mpart[b0 + (size_t)c * cap];
            s_w[c] = mc;
            s_l[c] = p.Lpart[b0 + (size_t)c * cap];
            M = fmaxf(M, mc);
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
        for (int c = tid; c < nlive; c += kWave) {
            const float mc = s_w[c];
            s_w[c] = mc == -INFINITY ? 0.0f : exp2f(mc - M);
        }
    }
    __syncthreads();
    if (tid == 0) {
        float den = 0.0f;
        for (int c = 0; c < nlive; ++c) den += s_w[c] * s_l[c];
        s_den = den;
    }
    __syncthreads();
    if (!has_dim) return;
    float num = 0.0f;
#pragma unroll
    for (int c = 0; c < kCombinePre; ++c)
        if (c < nlive) num += s_w[c] * pre[c];
    int c = kCombinePre;
    for (; c + 4 <= nlive; c += 4) {
        float o[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) o[u] = p.Opart[(b0 + (size_t)(c + u) * cap) * p.hd + dim];
#pragma unroll
        for (int u = 0; u < 4; ++u) num += s_w[c + u] * o[u];
    }
    for (; c < nlive; ++c) num += s_w[c] * p.Opart[(b0 + (size_t)c * cap) * p.hd + dim];
    put_act<P>(reinterpret_cast<T *>(p.O), act_plane(cap, p.d), act_idx<P>(row, h * p.hd + dim, p.d), num / s_den);
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

// Row table of the batch entries already listed in tab (seq[], nseq), from their control blocks:
// r0 prefix sums of the live block sizes (bounded by the row capacity cap), then one RowInfo per
// row. Called by a whole workgroup.
__device__ void plan_rows(Ctl *ctl, RowTab *tab, RowInfo *rows, int cap) {
    __shared__ int s_r0[kMaxSeqs], s_m[kMaxSeqs], s_L[kMaxSeqs], s_R;
    const int nseq = tab->nseq;
    if (threadIdx.x == 0) {
        int R = 0;
        for (int b = 0; b < nseq; ++b) {
            const Ctl *c = ctl + tab->seq[b];
            int m = c->m > 0 ? (c->m < kMaxBlock ? c->m : kMaxBlock) : 0;
            m = m < cap - R ? m : cap - R;
            tab->r0[b] = R;
            tab->m[b] = m;
            tab->L[b] = c->L;
            s_r0[b] = R;
            s_m[b] = m;
            s_L[b] = c->L;
            R += m;
        }
        tab->R = R;
        s_R = R;
    }
    __syncthreads();
    for (int row = threadIdx.x; row < s_R; row += blockDim.x) {
        int b = 0;
        while (b + 1 < nseq && row >= s_r0[b + 1]) ++b;  // the last entry starting at or before row
        const int i = row - s_r0[b];
        rows[row] = RowInfo{b, s_L[b] + i, ctl[tab->seq[b]].z[i], i};
    }
}

__global__ __launch_bounds__(256) void plan_kernel(PlanParams p) { plan_rows(p.ctl, p.tab, p.rows, p.cap); }

// Lay out the first block of a decode after the prefill, for batch entry blockIdx.x.
__global__ void decode_init_kernel(ScanParams p) {
    if (threadIdx.x != 0 || (int)blockIdx.x >= p.tab->nseq) return;
    const int seq = p.tab->seq[blockIdx.x];
    Ctl *c = p.ctl + seq;
    const int32_t *stream = p.stream ? p.stream + (size_t)seq * p.stream_stride : nullptr;
    c->mode = MODE_DECODE;
    c->e = 0;
    c->b0 = 0;
    c->nb = c->n < c->max_new ? c->n : c->max_new;
    c->steps = 0;
    c->rows = 0;
    c->blocks = 1;
    c->done = 0;
    c->err = 0;
    for (int i = 0; i <= kMaxBlock; ++i) c->hist[i] = 0;
    c->z[0] = c->pending;
    for (int j = 1; j < c->nb; ++j) c->z[j] = draw_guess(c, stream, j, 0);
    c->m = c->nb;
}

// Acceptance, commit, emit and the next block of one sequence, from its predictions c->pred
// (one thread).
__device__ void commit_and_next(Ctl *c, int m, int32_t *out, const int32_t *stream, int32_t *mlog, int32_t *rec) {
    for (int i = 0; i < (c->mode == MODE_PREFILL ? 1 : m); ++i)
        if (c->pred[i] < 0) {
            c->err |= 1;
            c->done = 1;
            c->m = 0;
            return;
        }
    if (c->mode == MODE_PREFILL) {  // every row is committed; pred[0] is the last row's argmax
        c->L += m;
        c->pending = c->pred[0];
        c->m = 0;
        return;
    }
    int a = 1;
    while (a < m && c->z[a] == c->pred[a - 1]) ++a;
    if (rec) {  // trajectory record header (its z and pred were written by the scan's threads)
        rec[0] = c->L;
        rec[1] = c->e;
        rec[2] = c->block_policy == 0 ? c->b0 : c->e;
        rec[3] = m;
        rec[4] = a;
    }
    c->L += a;
    c->a_last = a;
    if (mlog && c->mode == MODE_DECODE && c->steps < c->max_new) mlog[c->steps] = m;
    c->steps += 1;
    c->rows += m;
    c->hist[a] += 1;
    c->pending = c->pred[a - 1];
    if (c->mode != MODE_DECODE) {
        c->m = 0;
        return;
    }
    for (int k = 0; k < a; ++k) out[c->e + k] = c->z[k];
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
            for (int j = 1; j < newm; ++j) c->z[j] = draw_guess(c, stream, e + j, draw);
        } else {
            newm = c->b0 + c->nb - e;
            for (int j = 1; j < newm; ++j)
                c->z[j] = c->policy == 2 ? draw_guess(c, stream, e + j, draw) : c->pred[a - 1 + j];
        }
    } else {
        newm = (c->max_new - e) < n ? (c->max_new - e) : n;
        for (int j = 1; j < newm; ++j) {
            const int src = a - 1 + j;
            c->z[j] = (c->policy != 2 && src < m) ? c->pred[src] : draw_guess(c, stream, e + j, draw);
        }
    }
    c->z[0] = c->pending;
    c->m = newm;
}

// One workgroup per batch entry: the final argmax of each of its rows over the LM-head
// workgroups (16 threads per row take strided workgroups, then a 16-way tree; (max, lowest id)
// is exact, so the order is free), then commit_and_next. A prefill chunk needs only its last
// row. With one batch entry the workgroup also lays out the next row table.
__global__ __launch_bounds__(1024) void scan_commit_kernel(ScanParams p) {
    const int bi = blockIdx.x;
    const RowTab *tab = p.tab;
    if (bi >= tab->nseq) return;
    const int seq = tab->seq[bi];
    const int m = tab->m[bi], r0 = tab->r0[bi];
    Ctl *c = p.ctl + seq;
    const int tid = threadIdx.x;
    if (m > 0) {
        if (p.advance_only) {
            if (tid == 0) {
                c->L += m;
                c->m = 0;
            }
        } else {
            const bool prefill = c->mode == MODE_PREFILL;
            const int nrows = prefill ? 1 : m;            // <= 64
            const int rbase = r0 + (prefill ? m - 1 : 0);
            const int row = tid & 63, j = tid >> 6;
            float bv = -INFINITY;
            int bx = 0x7fffffff;
            int nan = 0;
            if (row < nrows) {
                for (int g0 = j; g0 < p.n_wg; g0 += 16 * 8) {
                    float v[8];
                    int ix[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        const int g = g0 + 16 * u;
                        ix[u] = g < p.n_wg ? p.pidx[(size_t)g * p.cap + rbase + row] : 0x7fffffff;
                        v[u] = g < p.n_wg ? p.pmax[(size_t)g * p.cap + rbase + row] : -INFINITY;
                    }
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        if (ix[u] < 0) nan = 1;
                        else if (v[u] > bv || (v[u] == bv && ix[u] < bx)) { bv = v[u]; bx = ix[u]; }
                    }
                }
            }
            __shared__ float s_v[1024];
            __shared__ int s_i[1024];
            __shared__ int s_nan[1024];
            s_v[tid] = bv;
            s_i[tid] = bx;
            s_nan[tid] = nan;
            __syncthreads();
            // this iteration's trajectory record (decode loops with recording on)
            int32_t *rec = (p.trace && c->mode == MODE_DECODE && c->steps < p.trace_cap)
                               ? p.trace + ((size_t)seq * p.trace_cap + c->steps) * kTraceStride
                               : nullptr;
            if (tid < nrows) {
                float best = s_v[tid];
                int i = s_i[tid], nn = s_nan[tid];
                for (int jj = 1; jj < 16; ++jj) {
                    const float ov = s_v[jj * 64 + tid];
                    const int oi = s_i[jj * 64 + tid];
                    nn |= s_nan[jj * 64 + tid];
                    if (ov > best || (ov == best && oi < i)) { best = ov; i = oi; }
                }
                const int pr = (nn || i == 0x7fffffff) ? -1 : i;
                c->pred[tid] = pr;
                if (rec) {
                    rec[5 + tid] = c->z[tid];
                    rec[5 + kMaxBlock + tid] = pr;
                }
            }
            __syncthreads();
            if (tid == 0)
                commit_and_next(c, m, p.out ? p.out + (size_t)seq * p.out_stride : nullptr,
                                p.stream ? p.stream + (size_t)seq * p.stream_stride : nullptr,
                                p.mlog ? p.mlog + (size_t)seq * p.out_stride : nullptr, rec);
        }
    }
    if (p.plan_inline) {
        __syncthreads();
        plan_rows(p.ctl, p.tab, p.rows, p.cap);
    }
}

// ------------------------------------------------------------------------------------------
// Weight repacking into the streaming tile layout. perm[r] is the logical source row of packed
// row r (-1: zero padding).
// ------------------------------------------------------------------------------------------
template <Prec P>
__global__ void repack_kernel(const void *src, const int32_t *perm, int K, int Ks, int n_tiles, uint8_t *dst) {
    using PT = PrecT<P>;
    using T = typename PT::T;
    const size_t tile = (size_t)blockIdx.x + (size_t)blockIdx.y * gridDim.x;  // = s * n_tiles + t
    if (tile >= (size_t)n_tiles * Ks) return;
    const int t = (int)(tile % n_tiles), s = (int)(tile / n_tiles);
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
// Grid: column workgroups (ceil(p.cols / (16 * NT))) x row tiles of 16 * RG rows (from row tile
// p.rt0) x K splits (E_LOGITS with p.kc > 0).
template <Prec P, int NT, int RG, int EP, int D = kGemmDepth, int W = kGemmWaves>
static hipError_t launch_gemm_t(const GemmParams &p, int row_tiles, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    constexpr int ROWS = 16 * RG, COLS = 16 * NT;
    static_assert(W * NT * 256 >= ROWS * COLS, "E_RESID reuses the reduction buffer");
    const size_t lds = (size_t)(W * NT * 256 + ROWS * (COLS + 1) + kMaxRows) * sizeof(float);
    auto kern = row_tiles > 1 ? gemm_kernel<P, NT, RG, EP, D, W, true> : gemm_kernel<P, NT, RG, EP, D, W, false>;
    GemmParams q = p;
    q.row_tiles = row_tiles;
    q.n_wg = (p.cols + COLS - 1) / COLS;  // the last workgroup may be ragged
    const int splits = EP == E_LOGITS && p.kc > 0 ? (p.Ks + p.kc - 1) / p.kc : 1;
    if (EP != E_LOGITS && p.kc != 0) return hipErrorInvalidValue;
    const dim3 grid(q.n_wg, row_tiles, splits);
    if (e0 || e1) {
        hipExtLaunchKernelGGL(kern, grid, dim3(W * kWave), lds, s, e0, e1, 0, q);
    } else {
        hipLaunchKernelGGL(kern, grid, dim3(W * kWave), lds, s, q);
    }
    return hipGetLastError();
}

template <Prec P, int RG>
static hipError_t launch_gemm_rg(GemmKind kind, const GemmParams &p, int row_tiles, hipStream_t s, hipEvent_t e0,
                                 hipEvent_t e1) {
    if (row_tiles > 1) {
        // More than 64 rows (measured at 160 and 512 rows, 7B): QKV and gate/up take 96-column
        // workgroups (two k-steps in flight), O and down 64-column workgroups (three k-steps in
        // flight). Row tiles past the iteration's rows exit at once, so a batched iteration
        // launched for its largest row count costs what its live rows cost.
        switch (kind) {
        case GEMM_QKV:
            return launch_gemm_t<P, 6, RG, E_QKV, 2>(p, row_tiles, s, e0, e1);
        case GEMM_O:
        case GEMM_DOWN:
            return launch_gemm_t<P, 4, RG, E_RESID, 3>(p, row_tiles, s, e0, e1);
        case GEMM_GATE_UP:
            return launch_gemm_t<P, 6, RG, E_SWIGLU, 2>(p, row_tiles, s, e0, e1);
        case GEMM_LM:
            return launch_gemm_t<P, kLmTiles, RG, E_ARGMAX, 3>(p, row_tiles, s, e0, e1);
        case GEMM_LOGITS:
            return launch_gemm_t<P, kLmTiles, RG, E_LOGITS, 3>(p, row_tiles, s, e0, e1);
        }
        return hipErrorInvalidValue;
    }
    switch (kind) {
    case GEMM_QKV:
        return launch_gemm_t<P, kNtQkv, RG, E_QKV>(p, row_tiles, s, e0, e1);
    case GEMM_O:
    case GEMM_DOWN:
        return launch_gemm_t<P, kNtResid, RG, E_RESID>(p, row_tiles, s, e0, e1);
    case GEMM_GATE_UP:
        return launch_gemm_t<P, kNtGateUp, RG, E_SWIGLU>(p, row_tiles, s, e0, e1);
    case GEMM_LM:
        return launch_gemm_t<P, kLmTiles, RG, E_ARGMAX>(p, row_tiles, s, e0, e1);
    case GEMM_LOGITS:
        return launch_gemm_t<P, kLmTiles, RG, E_LOGITS>(p, row_tiles, s, e0, e1);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemm(GemmKind kind, bool bf16, int rg, int row_tiles, const GemmParams &p, hipStream_t s,
                       hipEvent_t e0, hipEvent_t e1) {
    if (row_tiles < 1 || (row_tiles > 1 && rg != 4)) return hipErrorInvalidValue;
    if (bf16) {
        if (rg == 1) return launch_gemm_rg<Prec::BF16, 1>(kind, p, row_tiles, s, e0, e1);
        if (rg == 2) return launch_gemm_rg<Prec::BF16, 2>(kind, p, row_tiles, s, e0, e1);
        return launch_gemm_rg<Prec::BF16, 4>(kind, p, row_tiles, s, e0, e1);
    }
    if (rg == 1) return launch_gemm_rg<Prec::F32, 1>(kind, p, row_tiles, s, e0, e1);
    if (rg == 2) return launch_gemm_rg<Prec::F32, 2>(kind, p, row_tiles, s, e0, e1);
    return launch_gemm_rg<Prec::F32, 4>(kind, p, row_tiles, s, e0, e1);
}

hipError_t launch_embed(bool bf16, int rows, const EmbedParams &p, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    if (rows < 1 || rows > p.rr.cap) return hipErrorInvalidValue;  // every row entry read is within the table
    auto kern = bf16 ? embed_kernel<Prec::BF16> : embed_kernel<Prec::F32>;
    if (e0)
        hipExtLaunchKernelGGL(kern, dim3(rows), dim3(256), 0, s, e0, e1, 0, p);
    else
        hipLaunchKernelGGL(kern, dim3(rows), dim3(256), 0, s, p);
    return hipGetLastError();
}

template <Prec P, int HD>
static hipError_t launch_attn_hd(int rg, const AttnParams &p, int nch_launch, int nseq_launch, hipStream_t s,
                                 hipEvent_t e0, hipEvent_t e1) {
    if (p.nrb < 1 || (p.nrb > 1 && rg != 4)) return hipErrorInvalidValue;
    dim3 grid(nch_launch, p.n_heads, nseq_launch * p.nrb);
    auto kern = rg == 1 ? attn_partial_kernel<P, HD, 1>
                        : (rg == 2 ? attn_partial_kernel<P, HD, 2> : attn_partial_kernel<P, HD, 4>);
    if (e0)
        hipExtLaunchKernelGGL(kern, grid, dim3(kWave * rg), 0, s, e0, e1, 0, p);
    else
        hipLaunchKernelGGL(kern, grid, dim3(kWave * rg), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_attn(bool bf16, int rg, int nch_launch, int nseq_launch, const AttnParams &p, hipStream_t s,
                       hipEvent_t e0, hipEvent_t e1) {
    if (nseq_launch < 1 || nseq_launch > kMaxSeqs) return hipErrorInvalidValue;  // entries index the row table
    if (bf16) {
        switch (p.hd) {
        case 32: return launch_attn_hd<Prec::BF16, 32>(rg, p, nch_launch, nseq_launch, s, e0, e1);
        case 64: return launch_attn_hd<Prec::BF16, 64>(rg, p, nch_launch, nseq_launch, s, e0, e1);
        case 128: return launch_attn_hd<Prec::BF16, 128>(rg, p, nch_launch, nseq_launch, s, e0, e1);
        case 256: return launch_attn_hd<Prec::BF16, 256>(rg, p, nch_launch, nseq_launch, s, e0, e1);
        }
    } else {
        switch (p.hd) {
        case 16: return launch_attn_hd<Prec::F32, 16>(rg, p, nch_launch, nseq_launch, s, e0, e1);
        case 32: return launch_attn_hd<Prec::F32, 32>(rg, p, nch_launch, nseq_launch, s, e0, e1);
        case 64: return launch_attn_hd<Prec::F32, 64>(rg, p, nch_launch, nseq_launch, s, e0, e1);
        case 128: return launch_attn_hd<Prec::F32, 128>(rg, p, nch_launch, nseq_launch, s, e0, e1);
        }
    }
    return hipErrorInvalidValue;
}

template <Prec P, int HD>
static hipError_t launch_attn_fused_hd(int nrg, int nseq_launch, const AttnParams &p, hipStream_t s, hipEvent_t e0,
                                       hipEvent_t e1) {
    dim3 grid(p.n_heads * (HD / 16), nrg, nseq_launch);
    auto kern = attn_kernel<P, HD>;
    if (e0)
        hipExtLaunchKernelGGL(kern, grid, dim3(kAttnWaves * kWave), 0, s, e0, e1, 0, p);
    else
        hipLaunchKernelGGL(kern, grid, dim3(kAttnWaves * kWave), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_attn_fused(bool bf16, int nrg, int nseq_launch, const AttnParams &p, hipStream_t s, hipEvent_t e0,
                             hipEvent_t e1) {
    if (nseq_launch < 1 || nseq_launch > kMaxSeqs || nrg < 1) return hipErrorInvalidValue;
    if (bf16) {
        switch (p.hd) {
        case 32: return launch_attn_fused_hd<Prec::BF16, 32>(nrg, nseq_launch, p, s, e0, e1);
        case 64: return launch_attn_fused_hd<Prec::BF16, 64>(nrg, nseq_launch, p, s, e0, e1);
        case 128: return launch_attn_fused_hd<Prec::BF16, 128>(nrg, nseq_launch, p, s, e0, e1);
        }  // head_dim 256: two chunks of keys do not fit the registers; the two-kernel path
    } else {
        switch (p.hd) {
        case 16: return launch_attn_fused_hd<Prec::F32, 16>(nrg, nseq_launch, p, s, e0, e1);
        case 32: return launch_attn_fused_hd<Prec::F32, 32>(nrg, nseq_launch, p, s, e0, e1);
        case 64: return launch_attn_fused_hd<Prec::F32, 64>(nrg, nseq_launch, p, s, e0, e1);
        case 128: return launch_attn_fused_hd<Prec::F32, 128>(nrg, nseq_launch, p, s, e0, e1);
        }
    }
    return hipErrorInvalidValue;
}

hipError_t launch_attn_combine(bool bf16, int rows, const AttnParams &p, hipStream_t s, hipEvent_t e0,
                               hipEvent_t e1) {
    if (rows > p.rr.cap || p.hd > 256) return hipErrorInvalidValue;
    dim3 grid(p.n_heads, rows);
    const unsigned threads = p.hd < kWave ? (unsigned)kWave : (unsigned)p.hd;  // wave 0 reduces the maxima
    auto kern = bf16 ? attn_combine_kernel<Prec::BF16> : attn_combine_kernel<Prec::F32>;
    if (e0)
        hipExtLaunchKernelGGL(kern, grid, dim3(threads), 0, s, e0, e1, 0, p);
    else
        hipLaunchKernelGGL(kern, grid, dim3(threads), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_scan(int nseq_launch, const ScanParams &p, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    if (e0)
        hipExtLaunchKernelGGL(scan_commit_kernel, dim3(nseq_launch), dim3(1024), 0, s, e0, e1, 0, p);
    else
        hipLaunchKernelGGL(scan_commit_kernel, dim3(nseq_launch), dim3(1024), 0, s, p);
    return hipGetLastError();
}

static_assert(kMaxSeqs == 64, "SetupParams holds 64 entries");

// Host edits: entry b's block (or prefill chunk) of m[b] tokens, then the row table.
__global__ __launch_bounds__(256) void setup_kernel(SetupParams p) {
    __shared__ int s_r0[kMaxSeqs], s_L[kMaxSeqs];
    if (threadIdx.x == 0) {
        int R = 0;
        for (int b = 0; b < p.nseq; ++b) {
            Ctl *c = p.ctl + p.seq[b];
            if (p.set_L) {
                c->L = p.L;
                c->err = 0;
                c->done = 0;
            }
            c->mode = p.mode;
            c->m = p.m[b];
            if (p.mode != MODE_PREFILL)
                for (int i = 0; i < p.m[b]; ++i) c->z[i] = p.zin[(size_t)b * p.zstride + i];
            p.tab->seq[b] = p.seq[b];
            p.tab->r0[b] = R;
            p.tab->m[b] = p.m[b];
            p.tab->L[b] = c->L;
            s_r0[b] = R;
            s_L[b] = c->L;
            R += p.m[b];
        }
        p.tab->nseq = p.nseq;
        p.tab->R = R;
    }
    __syncthreads();
    for (int b = 0; b < p.nseq; ++b)
        for (int i = threadIdx.x; i < p.m[b]; i += blockDim.x)
            p.rows[s_r0[b] + i] = RowInfo{b, s_L[b] + i, p.zin[(size_t)b * p.zstride + i], i};
}

hipError_t launch_setup(const SetupParams &p, hipStream_t s) {
    hipLaunchKernelGGL(setup_kernel, dim3(1), dim3(256), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_decode_init(int nseq, const ScanParams &p, hipStream_t s) {
    hipLaunchKernelGGL(decode_init_kernel, dim3(nseq), dim3(kWave), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_plan(const PlanParams &p, hipStream_t s) {
    hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(256), 0, s, p);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void fill_weights_kernel(int kind, uint64_t key, double stdv, size_t n, void *out) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
        if (kind == 2) {
            static_cast<float *>(out)[i] = 1.0f;
            continue;
        }
        const uint64_t j = i >> 1;
        const uint64_t b1 = mix64(key ^ (2 * j)), b2 = mix64(key ^ (2 * j + 1));
        const double u1 = ((double)(b1 >> 11) + 1.0) * 0x1.0p-53;
        const double u2 = (double)(b2 >> 11) * 0x1.0p-53;
        const double r = sqrt(-2.0 * log(u1));
        const double a = 6.283185307179586476925286766559 * u2;
        const float x = (float)(stdv * ((i & 1) ? r * sin(a) : r * cos(a)));
        if (kind == 1)
            static_cast<uint16_t *>(out)[i] = f2bf(x);
        else
            static_cast<float *>(out)[i] = x;
    }
}

hipError_t launch_fill_weights(int kind, uint64_t key, double stdv, size_t n, void *out, hipStream_t s) {
    if (kind < 0 || kind > 2 || !out) return hipErrorInvalidValue;
    if (n == 0) return hipSuccess;
    const size_t blocks = std::min<size_t>((n + 255) / 256, 65536);
    hipLaunchKernelGGL(fill_weights_kernel, dim3((unsigned)blocks), dim3(256), 0, s, kind, key, stdv, n, out);
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
