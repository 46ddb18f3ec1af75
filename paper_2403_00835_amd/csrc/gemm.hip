// Weight-streaming GEMM of libcllm.so on gfx950 (CDNA4): the products of a Jacobi iteration
// (QKV, O, gate/up, down, LM head) with their fused epilogues, and the fp32-output product of
// the training loss head.
#include <hip/hip_ext.h>

#include <algorithm>
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

// LDS floats of gemm_kernel's body
template <int NT, int RG, int W>
__host__ __device__ constexpr int tile_lds_floats() {
    return W * NT * 256 + 16 * RG * (16 * NT + 1) + kMaxRows;
}

// The body of gemm_kernel for column group wg, row tile p.rt0 + rt and K range z (E_LOGITS with
// p.kc > 0); smem holds tile_lds_floats<NT, RG, W>() floats.
template <Prec P, int NT, int RG, int EP, int D, int W, bool MT>
__device__ __forceinline__ void gemm_tile_body(GemmParams p, int wg, int rt, int z, float *smem, int row0_at = -1) {
    static_assert(W == 8, "the K split and its reduction tree are defined for 8 waves");
    constexpr bool ROWSCALE = EP != E_RESID && EP != E_LOGITS;  // the product follows an RMSNorm
    constexpr int ROWS = 16 * RG, COLS = 16 * NT;
    if constexpr (EP == E_LOGITS) {
        if (p.kc > 0) {  // split K: k-steps [z kc, min((z + 1) kc, Ks)), partial products to plane z
            const int ks0 = z * p.kc;
            p.W += (size_t)ks0 * (p.cols >> 4) * kTileBytes;
            p.A = reinterpret_cast<const uint8_t *>(p.A) + (size_t)ks0 * kWave * 16;  // 16-byte lane vectors
            p.Ks = min(p.kc, p.Ks - ks0);
            p.Zout += (size_t)z * p.zstride;
        }
    }
    // This workgroup's row tile: rows [row0, row0 + ROWS) of the iteration (within the row
    // capacity; row0_at, when given, places it); m of them are live. A launch of one row tile
    // (MT false) always has live rows, so nothing waits for the row count before the first loads;
    // with several row tiles (MT) a tile with no live row exits first.
    const int row0 = row0_at >= 0 ? row0_at : (p.rt0 + rt) * ROWS;
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

// gemm_kernel's body for row tile rt of a launch (rows from (p.rt0 + rt) 16 RG on) with only as
// many 16-row groups as the tile has live rows (at most RG). A row's sums do not depend on the
// row groups computed beside it, so every row keeps its values, and a tile of few rows (a
// shrinking block, the last tile of a batched iteration) streams the weights with fewer operand
// rows and MFMAs. A one-tile launch (MT false) reads the row count before its first loads (the
// host knows only the block size, not the rows each queued iteration will have); a launch of
// several tiles reads it anyway, to let dead tiles exit. smem holds tile_lds_floats<NT, RG, W>()
// floats.
template <Prec P, int NT, int RG, int EP, int D, int W, bool MT>
__device__ __forceinline__ void gemm_tile_body_live(const GemmParams &p, int wg, int rt, int z, float *smem) {
    if constexpr (RG > 1) {
        const int row0 = (p.rt0 + rt) * 16 * RG;
        const int m = p.rr.tab->R - row0;
        if (m <= 16) return gemm_tile_body<P, NT, 1, EP, D, W, MT>(p, wg, 0, z, smem, row0);
        if constexpr (RG > 2) {
            if (m <= 32) return gemm_tile_body<P, NT, 2, EP, D, W, MT>(p, wg, 0, z, smem, row0);
        }
        if constexpr (RG > 3) {
            if (m <= 48) return gemm_tile_body<P, NT, 3, EP, D, W, MT>(p, wg, 0, z, smem, row0);
        }
    }
    gemm_tile_body<P, NT, RG, EP, D, W, MT>(p, wg, rt, z, smem);
}

template <Prec P, int NT, int RG, int EP, int D, int W, bool MT>
__global__ __launch_bounds__(W * kWave) void gemm_kernel(GemmParams p) {
    extern __shared__ float smem[];
    gemm_tile_body_live<P, NT, RG, EP, D, W, MT>(p, blockIdx.x, blockIdx.y, blockIdx.z, smem);
}

// ------------------------------------------------------------------------------------------
// Prompt GEMM (prefill passes, bf16): Y[rows x N] = A[rows x K] * W^T over the same packed
// operands, for workgroup tiles of 16 RG rows x 16 NT columns. The 8 waves form a WM x (8 / WM)
// grid over the tile and each accumulates its sub-tile over every k-step in order (one MFMA per
// plane, hi then lo). The operands of a k-step (2 RG activation blocks and NT weight tiles of
// 1 KiB each) are loaded once per workgroup from global memory straight into LDS (LDS DMA: no
// register round trip, no LDS write instructions), into a ring of NB buffers NB - 1 k-steps
// ahead, with a small LDS footprint so that two or three workgroups share a CU and hide each
// other's latency. A k-step's blocks are complete once this wave's DMA count has dropped to the
// later k-steps' loads (explicit vmcnt wait) and every wave has passed a barrier; the barrier is
// issued without the compiler's LDS fence (which would wait for every outstanding DMA), with
// compiler-only fences so no LDS access moves across it. The buffer a k-step refills was last
// read in the previous k-step, before that barrier. A row's reduction order depends only on K
// (and on the fixed K ranges of a split launch), never on the rows of a pass, so every prompt
// row gets the same values whatever the chunk size; the order differs from gemm_kernel's (which
// keeps eight k-step classes so decode rows are exact across row counts), so prompt rows always
// take this kernel. Epilogues and the RMSNorm row factor are gemm_kernel's.
// ------------------------------------------------------------------------------------------
template <int NT, int RG, int EP, int NB>
__host__ __device__ constexpr int prompt_dma_lds_floats() {
    constexpr int ROWS = 16 * RG, COLS = 16 * NT, BLK = 2 * RG + NT;
    constexpr int stage = NB * BLK * kWave * 4;
    constexpr int after = (EP == E_RESID ? ROWS * COLS : 0) + ROWS * (COLS + 1);
    return (stage > after ? stage : after) + ROWS;
}

template <int NT, int RG, int WM, int EP, int NB>
__global__ __launch_bounds__(kGemmWaves * kWave) void gemm_prompt_dma_kernel(GemmParams p) {
    constexpr Prec P = Prec::BF16;
    constexpr int W = kGemmWaves, WN = W / WM, RGW = RG / WM, NTW = NT / WN;
    constexpr int BLK = 2 * RG + NT, NLW = BLK / W;  // 1 KiB blocks per k-step, DMA loads per wave
    static_assert(RG % WM == 0 && NT % WN == 0 && BLK % W == 0 && NB >= 3, "tile split, ring depth");
    constexpr bool ROWSCALE = EP != E_RESID && EP != E_LOGITS;  // the product follows an RMSNorm
    constexpr int ROWS = 16 * RG, COLS = 16 * NT;
    // Workgroup L runs on XCD L % 8 (round-robin dispatch). Column group cg belongs to XCD cg % 8,
    // and each XCD takes its column groups in turn with their row tiles consecutively, so the row
    // tiles of a column group run together and read its weights once from HBM into that XCD's L2.
    const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
    const int wg = (slot / p.row_tiles) * 8 + xcd, row0 = (slot % p.row_tiles) * ROWS;
    request_together(p.W, p.A, p.ssq, p.Ks, p.cols, p.lda, p.rr.cap, p.T, p.n_wg);
    const int m = p.rr.tab->R - row0;
    if (m <= 0 || wg >= p.n_wg) return;
    const int rg0 = row0 >> 4, t0 = wg * NT;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = w / WN, wn = w % WN;
    // E_LOGITS with p.kc > 0: grid y takes k-steps [y kc, min((y + 1) kc, Ks)) and writes its
    // partial products to plane y
    int Ks = p.Ks, ks0 = 0;
    if constexpr (EP == E_LOGITS) {
        if (p.kc > 0) {
            ks0 = blockIdx.y * p.kc;
            Ks = min(p.kc, p.Ks - ks0);
            p.Zout += (size_t)blockIdx.y * p.zstride;
        }
    }

    extern __shared__ float smem[];
    u32x4 *s_stage = reinterpret_cast<u32x4 *>(smem);  // [NB][BLK][64] during the main loop
    float *s_red = smem;                               // then epilogue scratch (E_RESID) ...
    float *s_tile = smem + (EP == E_RESID ? ROWS * COLS : 0);  // ... and the output tile
    float *s_inv = smem + prompt_dma_lds_floats<NT, RG, EP, NB>() - ROWS;  // row factors (apart)

    f32x4 sq_pre[2];
    if constexpr (ROWSCALE) row_factor_preload<W>(p, row0, tid, sq_pre);

    // This wave's blocks b = w + i W of every k-step: block b < 2 RG is activation plane b / RG,
    // row group b % RG; block 2 RG + j is weight tile t0 + j (clamped). A k-step advances an
    // activation block by 64 vectors and a weight block by one k-step of tiles.
    const int tiles = p.cols >> 4, ks_a = p.lda / PrecT<P>::KSTEP;
    const u32x4 *src[NLW];
    int adv[NLW];
#pragma unroll
    for (int i = 0; i < NLW; ++i) {
        const int b = w + i * W;
        if (b < 2 * RG) {
            const uint16_t *A = reinterpret_cast<const uint16_t *>(p.A) + (b / RG) * act_plane(p.rr.cap, p.lda);
            src[i] = reinterpret_cast<const u32x4 *>(A + (size_t)(rg0 + b % RG) * ks_a * kWave * 8) + lane;
            adv[i] = kWave;
        } else {
            src[i] = reinterpret_cast<const u32x4 *>(p.W + (size_t)min(t0 + b - 2 * RG, tiles - 1) * kTileBytes) + lane;
            adv[i] = tiles * kWave;
        }
        src[i] += (size_t)ks0 * adv[i];  // the first k-step of this workgroup's K range
    }
    // k-step s into ring buffer s % NB; past the last k-step a harmless reload of it
    auto issue = [&](int s) {
        const size_t ss = (size_t)min(s, Ks - 1);
        u32x4 *buf = s_stage + (size_t)(s % NB) * BLK * kWave;
#pragma unroll
        for (int i = 0; i < NLW; ++i)
            __builtin_amdgcn_global_load_lds(static_cast<const void *>(src[i] + ss * adv[i]),
                                             (__attribute__((address_space(3))) void *)(buf + (size_t)(w + i * W) * kWave),
                                             16, 0, 0);
    };
    f32x4 acc[RGW][NTW];
#pragma unroll
    for (int r = 0; r < RGW; ++r)
#pragma unroll
        for (int j = 0; j < NTW; ++j) acc[r][j] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
    for (int q = 0; q < NB - 1; ++q) issue(q);
    for (int s = 0; s < Ks; ++s) {
        wait_vm<(NB - 2) * NLW>();  // this wave's blocks of k-step s have landed
        barrier_no_fence();         // every wave's; buffer (s - 1) % NB has no reader left
        issue(s + NB - 1);
        const u32x4 *bp = s_stage + (size_t)(s % NB) * BLK * kWave + lane;
        u32x4 a[2][RGW], b[NTW];
#pragma unroll
        for (int pl = 0; pl < 2; ++pl)
#pragma unroll
            for (int r = 0; r < RGW; ++r) a[pl][r] = bp[(pl * RG + wm * RGW + r) * kWave];
#pragma unroll
        for (int j = 0; j < NTW; ++j) b[j] = bp[(2 * RG + wn * NTW + j) * kWave];
#pragma unroll
        for (int pl = 0; pl < 2; ++pl)
#pragma unroll
            for (int r = 0; r < RGW; ++r)
#pragma unroll
                for (int j = 0; j < NTW; ++j) acc[r][j] = mfma_kstep<P>(a[pl][r], b[j], acc[r][j]);
    }
    wait_vm<0>();  // the trailing reloads have landed before the buffers are reused
    __syncthreads();

    if constexpr (ROWSCALE) row_factor_reduce<W, ROWS>(p, row0, tid, sq_pre, s_inv);
    __syncthreads();
    // C layout of a 16 x 16 tile: lane l, register v -> row 4 (l / 16) + v, column l % 16
#pragma unroll
    for (int r = 0; r < RGW; ++r)
#pragma unroll
        for (int j = 0; j < NTW; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = 16 * (wm * RGW + r) + 4 * (lane >> 4) + v;
                float x = acc[r][j][v];
                if constexpr (ROWSCALE) x *= s_inv[row];
                s_tile[row * (COLS + 1) + 16 * (wn * NTW + j) + (lane & 15)] = x;
            }
    __syncthreads();
    gemm_epilogue<P, NT, RG, EP, W>(p, s_tile, s_red, row0, m, wg, tid, lane, w);
}

// ------------------------------------------------------------------------------------------
// Row-tiled decode GEMM (iterations of more than 64 rows, bf16): workgroup tiles of 64 rows x
// 16 NT columns with the operand blocks brought into LDS by DMA (as gemm_prompt_dma_kernel, NB
// buffers, NB - 1 k-steps in flight) and gemm_kernel's reduction order, so that every row gets
// the bits a one-tile iteration gives it (batched, AR and Jacobi decoding stay bit-identical):
// k-step k is accumulated into the set of its class k % 8 (from zero, the hi then the lo MFMA, in
// increasing k, as wave k % 8 of gemm_kernel accumulates it), and the eight class sums are folded
// at the end in gemm_kernel's tree ((x0 + x4) + (x2 + x6)) + ((x1 + x5) + (x3 + x7)). The RMSNorm
// row factor and the epilogues are gemm_kernel's. With p.kc > 0 (E_LOGITS) grid z splits K into
// ranges of kc k-steps, the classes of a range counted from its first k-step, as gemm_kernel
// splits it.
// ------------------------------------------------------------------------------------------
// tiles (16 columns) per workgroup and ring depth of the row-tiled products (measured at the
// LLaMA-2-7B shape, 96 to 512 rows; QKV and O stay faster on gemm_kernel)
constexpr int kRowsNtGateUp = 12, kRowsNbGateUp = 4;
constexpr int kRowsNtDown = 8, kRowsNbDown = 4;

template <int NT, int EP, int NB>
__host__ __device__ constexpr int rows_lds_floats() {
    constexpr int RG = 4, ROWS = 16 * RG, COLS = 16 * NT, BLK = 2 * RG + NT;
    constexpr int stage = NB * BLK * kWave * 4;
    constexpr int after = (EP == E_RESID ? ROWS * COLS : 0) + ROWS * (COLS + 1);
    return (stage > after ? stage : after) + ROWS;
}

// The row-tiled product of one tile of 16 RGT live rows (row0 on, m of them live) over a WM x
// (8 / WM) wave grid: eight class sums per output folded in gemm_kernel's tree, its row factor
// and epilogue. smem holds rows_lds_floats<NT, EP, NB>() floats (the launch's 64-row tile).
template <int RGT, int WM, int NT, int EP, int NB>
__device__ __forceinline__ void rows_tile_body(const GemmParams &p, int wg, int row0, int m, float *smem) {
    constexpr Prec P = Prec::BF16;
    constexpr int W = kGemmWaves, WN = W / WM, RGW = RGT / WM, NTW = NT / WN;
    constexpr int BLK = 2 * RGT + NT;
    static_assert(RGT % WM == 0 && NT % WN == 0 && NB >= 3, "tile split, ring depth");
    constexpr bool ROWSCALE = EP != E_RESID && EP != E_LOGITS;
    constexpr int ROWS = 16 * RGT, COLS = 16 * NT;
    const int rg0 = row0 >> 4, t0 = wg * NT;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = w / WN, wn = w % WN;
    const int Ks = p.Ks;

    u32x4 *s_stage = reinterpret_cast<u32x4 *>(smem);  // [NB][BLK][64] during the main loop
    float *s_red = smem;
    float *s_tile = smem + (EP == E_RESID ? ROWS * COLS : 0);
    float *s_inv = smem + rows_lds_floats<NT, EP, NB>() - kMaxRows;

    f32x4 sq_pre[2];
    if constexpr (ROWSCALE) row_factor_preload<W>(p, row0, tid, sq_pre);

    // DMA blocks of a k-step: block b < 2 RGT is activation plane b / RGT, row group b % RGT;
    // block 2 RGT + j is weight tile t0 + j (clamped; its columns are never written). Wave w
    // issues blocks w, w + W, ... (NLW of them; where the last round has no block for a wave, it
    // loads the last block again into its place), so every wave has the same number of loads in
    // flight.
    constexpr int NLW = (BLK + W - 1) / W;
    const int tiles = p.cols >> 4, ks_a = p.lda / PrecT<P>::KSTEP;
    const u32x4 *src[NLW];
    int adv[NLW], dst[NLW];
#pragma unroll
    for (int i = 0; i < NLW; ++i) {
        const int b = min(w + i * W, BLK - 1);
        dst[i] = b;
        if (b < 2 * RGT) {
            const uint16_t *A = reinterpret_cast<const uint16_t *>(p.A) + (b / RGT) * act_plane(p.rr.cap, p.lda);
            src[i] = reinterpret_cast<const u32x4 *>(A + (size_t)(rg0 + b % RGT) * ks_a * kWave * 8) + lane;
            adv[i] = kWave;
        } else {
            src[i] = reinterpret_cast<const u32x4 *>(p.W + (size_t)min(t0 + b - 2 * RGT, tiles - 1) * kTileBytes) + lane;
            adv[i] = tiles * kWave;
        }
    }
    auto issue = [&](int s, int buf) {  // k-step s (< Ks) into ring buffer buf
        u32x4 *bb = s_stage + (size_t)buf * BLK * kWave;
#pragma unroll
        for (int i = 0; i < NLW; ++i)
            __builtin_amdgcn_global_load_lds(static_cast<const void *>(src[i] + (size_t)s * adv[i]),
                                             (__attribute__((address_space(3))) void *)(bb + (size_t)dst[i] * kWave),
                                             16, 0, 0);
    };
    // one accumulator set per class: k-step k goes to set k % 8, the k-steps in increasing order
    f32x4 acc[8][RGW][NTW];
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int r = 0; r < RGW; ++r)
#pragma unroll
            for (int j = 0; j < NTW; ++j) acc[c][r][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // past the last k-step the ring reloads k-step Ks - 1 (harmless, never computed)
#pragma unroll
    for (int q = 0; q < NB - 1; ++q) issue(min(q, Ks - 1), q);
    int buf = 0;  // ring buffer of the k-step being computed
    for (int k0 = 0; k0 < Ks; k0 += 8) {
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const int k = k0 + c;
            if (k < Ks) {  // uniform over the workgroup
                wait_vm<(NB - 2) * NLW>();  // this wave's blocks of k-step k have landed
                barrier_no_fence();         // every wave's; the buffer refilled next has no reader left
                issue(min(k + NB - 1, Ks - 1), buf == 0 ? NB - 1 : buf - 1);
                const u32x4 *bp = s_stage + (size_t)buf * BLK * kWave + lane;
                u32x4 a[2][RGW], b[NTW];
#pragma unroll
                for (int pl = 0; pl < 2; ++pl)
#pragma unroll
                    for (int r = 0; r < RGW; ++r) a[pl][r] = bp[(pl * RGT + wm * RGW + r) * kWave];
#pragma unroll
                for (int j = 0; j < NTW; ++j) b[j] = bp[(2 * RGT + wn * NTW + j) * kWave];
#pragma unroll
                for (int pl = 0; pl < 2; ++pl)
#pragma unroll
                    for (int r = 0; r < RGW; ++r)
#pragma unroll
                        for (int j = 0; j < NTW; ++j) acc[c][r][j] = mfma_kstep<P>(a[pl][r], b[j], acc[c][r][j]);
                buf = buf == NB - 1 ? 0 : buf + 1;
            }
        }
    }
    wait_vm<0>();  // the trailing reloads have landed before the buffers are reused
    __syncthreads();

    if constexpr (ROWSCALE) row_factor_reduce<W, ROWS>(p, row0, tid, sq_pre, s_inv);
    __syncthreads();
    // gemm_kernel's tree over the class sums, then its row factor
#pragma unroll
    for (int r = 0; r < RGW; ++r)
#pragma unroll
        for (int j = 0; j < NTW; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = 16 * (wm * RGW + r) + 4 * (lane >> 4) + v;
                float x = ((acc[0][r][j][v] + acc[4][r][j][v]) + (acc[2][r][j][v] + acc[6][r][j][v])) +
                          ((acc[1][r][j][v] + acc[5][r][j][v]) + (acc[3][r][j][v] + acc[7][r][j][v]));
                if constexpr (ROWSCALE) x *= s_inv[row];
                s_tile[row * (COLS + 1) + 16 * (wn * NTW + j) + (lane & 15)] = x;
            }
    __syncthreads();
    gemm_epilogue<P, NT, RGT, EP, W>(p, s_tile, s_red, row0, m, wg, tid, lane, w);
}

// An iteration of at most 64 rows (one row tile; the row count is known only on the device) takes
// gemm_kernel's body with NT_T tiles per workgroup and D_T k-steps in flight instead: its column
// groups are narrower, so more workgroups share the work (one row tile of the row-tiled kernel
// would occupy fewer than half the CUs). The last live tile of a longer iteration runs only its
// live 16-row groups.
template <int NT, int EP, int NB, int NT_T, int D_T>
__global__ __launch_bounds__(kGemmWaves * kWave) void gemm_rows_kernel(GemmParams p) {
    constexpr Prec P = Prec::BF16;
    constexpr int RG = 4, W = kGemmWaves;
    constexpr int ROWS = 16 * RG;
    extern __shared__ float smem[];
    request_together(p.rr.tab, p.cols, p.rt0);
    if (p.rr.tab->R - p.rt0 * ROWS <= ROWS) {
        const int nwt = (p.cols + 16 * NT_T - 1) / (16 * NT_T);
        if ((int)blockIdx.x < nwt) gemm_tile_body_live<P, NT_T, RG, EP, D_T, W, true>(p, blockIdx.x, 0, blockIdx.z, smem);
        return;
    }
    if constexpr (EP == E_LOGITS) {
        if (p.kc > 0) {  // split K as gemm_kernel does
            const int ks0 = blockIdx.z * p.kc;
            p.W += (size_t)ks0 * (p.cols >> 4) * kTileBytes;
            p.A = reinterpret_cast<const uint8_t *>(p.A) + (size_t)ks0 * kWave * 16;
            p.Ks = min(p.kc, p.Ks - ks0);
            p.Zout += (size_t)blockIdx.z * p.zstride;
        }
    }
    // Column groups on XCDs in turn, the live row tiles of a column group consecutive on one XCD
    // (its L2 serves the weight tiles to all of them). The launch covers its largest row count; the
    // live row tiles (from the device row table) take the first workgroups of each XCD, so the
    // workgroups past them, which exit at once, are dispatched last.
    request_together(p.W, p.A, p.ssq, p.Ks, p.cols, p.lda, p.rr.cap, p.T, p.n_wg, p.row_tiles);
    const int live = min(p.row_tiles, (p.rr.tab->R - p.rt0 * ROWS + ROWS - 1) / ROWS);
    const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
    const int wg = (slot / live) * 8 + xcd, row0 = (p.rt0 + slot % live) * ROWS;
    if (wg >= p.n_wg) return;
    const int m = p.rr.tab->R - row0;
    // 16-row groups of this tile with live rows (every row's values are the same whatever the
    // tile's row groups and wave grid); one or three groups take a one-row wave grid, which needs
    // NT a multiple of the 8 waves
    if constexpr (NT % W == 0) {
        if (m <= 16) return rows_tile_body<1, 1, NT, EP, NB>(p, wg, row0, m, smem);
        if (m <= 32) return rows_tile_body<2, 2, NT, EP, NB>(p, wg, row0, m, smem);
        if (m <= 48) return rows_tile_body<3, 1, NT, EP, NB>(p, wg, row0, m, smem);
    } else {
        if (m <= 32) return rows_tile_body<2, 2, NT, EP, NB>(p, wg, row0, m, smem);
    }
    rows_tile_body<4, 2, NT, EP, NB>(p, wg, row0, m, smem);
}

template <int NT, int EP, int NB, int NT_T, int D_T>
static hipError_t launch_rows_t(const GemmParams &p, int row_tiles, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    constexpr int COLS = 16 * NT;
    constexpr int lds_rows = rows_lds_floats<NT, EP, NB>(), lds_tile = tile_lds_floats<NT_T, 4, kGemmWaves>();
    const size_t lds = (size_t)(lds_rows > lds_tile ? lds_rows : lds_tile) * sizeof(float);
    if (row_tiles < 1 || (p.rt0 + row_tiles) * 64 > p.rr.cap || p.lda % 32 != 0 || p.cols % 16 != 0)
        return hipErrorInvalidValue;
    if (EP != E_LOGITS && p.kc != 0) return hipErrorInvalidValue;
    GemmParams q = p;
    q.n_wg = (p.cols + COLS - 1) / COLS;
    q.row_tiles = row_tiles;
    const int splits = EP == E_LOGITS && p.kc > 0 ? (p.Ks + p.kc - 1) / p.kc : 1;
    const int n_tile = (p.cols + 16 * NT_T - 1) / (16 * NT_T);  // column groups of the one-tile body
    const dim3 grid((unsigned)std::max((q.n_wg + 7) / 8 * 8 * row_tiles, n_tile), 1, (unsigned)splits);
    auto kern = gemm_rows_kernel<NT, EP, NB, NT_T, D_T>;
    if (e0 || e1)
        hipExtLaunchKernelGGL(kern, grid, dim3(kGemmWaves * kWave), lds, s, e0, e1, 0, q);
    else
        hipLaunchKernelGGL(kern, grid, dim3(kGemmWaves * kWave), lds, s, q);
    return hipGetLastError();
}

// ------------------------------------------------------------------------------------------
// Class-pair K split of the decode GEMM (bf16, iterations of more than 64 rows). gemm_kernel's
// tree ((x0 + x4) + (x2 + x6)) + ((x1 + x5) + (x3 + x7)) over the eight k-step class sums equals
// (t0 + t2) + (t1 + t3) with t_c = x_c + x_(c+4). Grid z = c in {0, 1, 2, 3}: a workgroup walks
// the k-steps k = c (mod 4) in increasing order and accumulates those with k = c (mod 8) into one
// set and those with k = c + 4 (mod 8) into another (from zero, the hi then the lo MFMA, as wave
// k % 8 of gemm_kernel accumulates them), then writes t_c of its 16 RGT x 16 NT tile, fp32, to
// plane c of p.spart; gemm_split_reduce_kernel forms (t0 + t2) + (t1 + t3), applies the RMSNorm
// row factor and runs gemm_kernel's epilogue. Every row therefore gets the bits of a one-tile
// iteration. Two accumulator sets instead of eight allow workgroup tiles four times larger (each
// k-step's operand rows and weight tiles, brought into LDS by DMA through a ring of NB buffers,
// serve more outputs), and the four K quarters are four times finer units of work. An iteration
// whose live rows fit one 64-row tile (known only on the device) takes gemm_kernel's body with
// NT_T tiles per workgroup and D_T k-steps in flight inside the split launch, and the reduction
// launch then has nothing to do.
//
// p.spart, plane c: [row group of 16 rows][16-column tile][lane][4] fp32 in the MFMA's C layout
// (lane l, register v: row 4 (l / 16) + v, column l % 16 of the tile), row capacity x p.cols
// floats per plane.
// ------------------------------------------------------------------------------------------
// 16-column tiles per workgroup and ring depth of the split products (64-row tiles; measured at
// the LLaMA-2-7B shape, 160 and 512 rows: gate/up 74.6 / 195 us, QKV 45.0 / 100 us before the
// reduction; O is no faster than gemm_kernel once its reduction is added)
constexpr int kSplitNtQkv = 16, kSplitNbQkv = 3, kSplitNtGateUp = 16, kSplitNbGateUp = 3;
constexpr int kSplitNtLm = 16, kSplitNbLm = 3;

template <int RGT, int NT, int NB>
__host__ __device__ constexpr int split_lds_floats() {
    return NB * (2 * RGT + NT) * kWave * 4;
}

// The class-pair product of one tile of 16 RGT live rows (row0 on): the k-steps c, c + 4, ... into
// two accumulator sets over a WM x (8 / WM) wave grid, t_c written to plane c of p.spart.
// smem holds split_lds_floats<4, NT, NB>() floats (the launch's 64-row tile).
template <int RGT, int WM, int NT, int NB>
__device__ __forceinline__ void split_tile_body(const GemmParams &p, int c, int wg, int row0, float *smem) {
    constexpr Prec P = Prec::BF16;
    constexpr int W = kGemmWaves, WN = W / WM, RGW = RGT / WM, NTW = NT / WN;
    constexpr int BLK = 2 * RGT + NT, NLW = (BLK + W - 1) / W;
    static_assert(RGT % WM == 0 && NT % WN == 0 && NB >= 3, "tile split, ring depth");
    const int rg0 = row0 >> 4, t0 = wg * NT;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = w / WN, wn = w % WN;
    const int nq = (p.Ks - c + 3) >> 2;  // k-steps c, c + 4, ... below Ks (the launcher has Ks >= 4)
    const int last = c + 4 * (nq - 1);

    u32x4 *s_stage = reinterpret_cast<u32x4 *>(smem);  // [NB][BLK][64]
    // DMA blocks of a k-step: block b < 2 RGT is activation plane b / RGT, row group b % RGT; block
    // 2 RGT + j is weight tile t0 + j (clamped; its columns are never written). Wave w issues blocks
    // w, w + W, ... (NLW of them; where the last round has no block for a wave, it loads the last
    // block again into its place), so every wave has the same number of loads in flight.
    const int tiles = p.cols >> 4, ks_a = p.lda / PrecT<P>::KSTEP;
    const u32x4 *src[NLW];
    int adv[NLW], dst[NLW];
#pragma unroll
    for (int i = 0; i < NLW; ++i) {
        const int b = min(w + i * W, BLK - 1);
        dst[i] = b;
        if (b < 2 * RGT) {
            const uint16_t *A = reinterpret_cast<const uint16_t *>(p.A) + (b / RGT) * act_plane(p.rr.cap, p.lda);
            src[i] = reinterpret_cast<const u32x4 *>(A + (size_t)(rg0 + b % RGT) * ks_a * kWave * 8) + lane;
            adv[i] = kWave;
        } else {
            src[i] = reinterpret_cast<const u32x4 *>(p.W + (size_t)min(t0 + b - 2 * RGT, tiles - 1) * kTileBytes) + lane;
            adv[i] = tiles * kWave;
        }
    }
    auto issue = [&](int k, int buf) {  // k-step k (< Ks) into ring buffer buf
        u32x4 *bb = s_stage + (size_t)buf * BLK * kWave;
#pragma unroll
        for (int i = 0; i < NLW; ++i)
            __builtin_amdgcn_global_load_lds(static_cast<const void *>(src[i] + (size_t)k * adv[i]),
                                             (__attribute__((address_space(3))) void *)(bb + (size_t)dst[i] * kWave),
                                             16, 0, 0);
    };
    f32x4 acc[2][RGW][NTW];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int r = 0; r < RGW; ++r)
#pragma unroll
            for (int j = 0; j < NTW; ++j) acc[h][r][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // past the last k-step the ring reloads the last one (harmless, never computed)
#pragma unroll
    for (int q = 0; q < NB - 1; ++q) issue(min(c + 4 * q, last), q);
    int buf = 0;  // ring buffer of the k-step being computed
    for (int q0 = 0; q0 < nq; q0 += 2) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {  // k-step c + 4 (q0 + h): class c for h = 0, c + 4 for h = 1
            const int q = q0 + h;
            if (q < nq) {  // uniform over the workgroup
                wait_vm<(NB - 2) * NLW>();  // this wave's blocks of the k-step have landed
                barrier_no_fence();         // every wave's; the buffer refilled next has no reader left
                issue(min(c + 4 * (q + NB - 1), last), buf == 0 ? NB - 1 : buf - 1);
                const u32x4 *bp = s_stage + (size_t)buf * BLK * kWave + lane;
                u32x4 a[2][RGW], b[NTW];
#pragma unroll
                for (int pl = 0; pl < 2; ++pl)
#pragma unroll
                    for (int r = 0; r < RGW; ++r) a[pl][r] = bp[(pl * RGT + wm * RGW + r) * kWave];
#pragma unroll
                for (int j = 0; j < NTW; ++j) b[j] = bp[(2 * RGT + wn * NTW + j) * kWave];
#pragma unroll
                for (int pl = 0; pl < 2; ++pl)
#pragma unroll
                    for (int r = 0; r < RGW; ++r)
#pragma unroll
                        for (int j = 0; j < NTW; ++j) acc[h][r][j] = mfma_kstep<P>(a[pl][r], b[j], acc[h][r][j]);
                buf = buf == NB - 1 ? 0 : buf + 1;
            }
        }
    }
    wait_vm<0>();  // the trailing reloads have landed before the workgroup ends

    float *Z = p.spart + (size_t)c * p.rr.cap * p.cols;
#pragma unroll
    for (int r = 0; r < RGW; ++r)
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
            const int t = t0 + wn * NTW + j;
            if (t < tiles) {
                f32x4 v;
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = acc[0][r][j][e] + acc[1][r][j][e];
                *reinterpret_cast<f32x4 *>(Z + (((size_t)(rg0 + wm * RGW + r) * tiles + t) * kWave + lane) * 4) = v;
            }
        }
}

// The split product of a launch of several 64-row tiles, whatever the rows the iteration turns
// out to have (known only on the device): one that fits one tile takes the same path (the same
// values as gemm_kernel's). The kernel keeps to 128 registers (at least four waves per SIMD), so
// two workgroups share a CU.
template <int NT, int NB, int EP>
__global__ __launch_bounds__(kGemmWaves * kWave, 4) void gemm_split_kernel(GemmParams p) {
    constexpr int W = kGemmWaves;
    constexpr int ROWS = kMaxRows;
    extern __shared__ float smem[];
    // Column groups on XCDs in turn, the live row tiles of a column group consecutive on one XCD;
    // the launch covers its largest row count, the live row tiles take the first workgroups of
    // each XCD and the others exit at once.
    constexpr bool ROWSCALE = EP != E_RESID && EP != E_LOGITS;
    request_together(p.rr.tab, p.cols, p.rt0, p.W, p.A, p.Ks, p.lda, p.rr.cap, p.n_wg, p.row_tiles, p.spart, p.ssq,
                     p.T);
    const int R = p.rr.tab->R;
    if (R - p.rt0 * ROWS <= 0) return;
    const int live = min(p.row_tiles, (R - p.rt0 * ROWS + ROWS - 1) / ROWS);
    const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
    // XCD x takes class pair x % 4 and every other column group from x / 4
    const int c = xcd & 3, wg = (slot / live) * 2 + (xcd >> 2);
    const int row0 = (p.rt0 + slot % live) * ROWS;
    if (wg >= p.n_wg) return;
    const int tid = threadIdx.x;
    // one workgroup per row tile also computes the tile's RMSNorm row factors for the reduction
    const bool factors = ROWSCALE && wg == 0 && c == 0;
    f32x4 sq_pre[2];
    if (factors) row_factor_preload<W>(p, row0, tid, sq_pre);

    // The last live tile runs only its live 16-row groups (rows past the iteration's rows have
    // no partials; the reduction writes nothing for them). Every row's t_c is the same whatever
    // the tile's row groups and wave grid; one or three groups take a one-row wave grid, which
    // needs NT a multiple of the 8 waves.
    const int mt = R - row0;
    if constexpr (NT % W == 0) {
        if (mt <= 16)
            split_tile_body<1, 1, NT, NB>(p, c, wg, row0, smem);
        else if (mt <= 32)
            split_tile_body<2, 2, NT, NB>(p, c, wg, row0, smem);
        else if (mt <= 48)
            split_tile_body<3, 1, NT, NB>(p, c, wg, row0, smem);
        else
            split_tile_body<4, 2, NT, NB>(p, c, wg, row0, smem);
    } else {
        if (mt <= 32)
            split_tile_body<2, 2, NT, NB>(p, c, wg, row0, smem);
        else
            split_tile_body<4, 2, NT, NB>(p, c, wg, row0, smem);
    }

    if (factors) {  // uniform over the workgroup
        __syncthreads();  // every wave is past its last read of the ring
        float *s_inv = smem;
        row_factor_reduce<W, ROWS>(p, row0, tid, sq_pre, s_inv);
        __syncthreads();
        if (tid < ROWS) p.sinv[row0 + tid] = s_inv[tid];
    }
}

// (t0 + t2) + (t1 + t3) of the class-pair partials for a 64-row tile x 16 NT columns, the RMSNorm
// row factor (computed once per row tile by the split launch) and gemm_kernel's epilogue. Grid: column groups x row tiles (from p.rt0); row tiles
// past the iteration's rows exit.
template <int NT, int EP>
__host__ __device__ constexpr int split_reduce_lds_floats() {
    constexpr int ROWS = kMaxRows, COLS = 16 * NT;
    return (EP == E_RESID ? ROWS * COLS : 0) + ROWS * (COLS + 1) + ROWS;
}

template <int NT, int EP>
__global__ __launch_bounds__(kGemmWaves * kWave) void gemm_split_reduce_kernel(GemmParams p) {
    constexpr Prec P = Prec::BF16;
    constexpr int W = kGemmWaves, RG = kMaxRows / 16, ROWS = kMaxRows, COLS = 16 * NT;
    constexpr int NV = RG * NT * kWave / (W * kWave);  // 16-byte vectors per thread and plane
    static_assert((RG * NT) % W == 0, "every thread takes the same number of vectors");
    constexpr bool ROWSCALE = EP != E_RESID && EP != E_LOGITS;
    extern __shared__ float smem[];
    const int wg = blockIdx.x, row0 = (p.rt0 + blockIdx.y) * ROWS;
    request_together(p.rr.tab, p.spart, p.cols, p.rr.cap, p.sinv, p.rt0);
    const int m = p.rr.tab->R - row0;
    if (m <= 0) return;  // a row tile past the iteration's rows
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    float *s_red = smem;                                       // epilogue scratch (E_RESID)
    float *s_tile = smem + (EP == E_RESID ? ROWS * COLS : 0);  // ROWS x (COLS + 1)
    float *s_inv = s_tile + ROWS * (COLS + 1);                 // ROWS
    const int tiles = p.cols >> 4, t0 = wg * NT, rg0 = row0 >> 4;
    const size_t plane = (size_t)p.rr.cap * p.cols;
    // vector u = tid + i W 64: row group (u / 64) / NT, tile (u / 64) % NT, lane u % 64; row
    // groups past the iteration's rows (the split launch wrote no partials there; their rows are
    // not written out) load nothing
    f32x4 z[NV][4];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int u = tid + i * W * kWave, blk = u >> 6;
        const int r = blk / NT, t = min(t0 + blk % NT, tiles - 1);
        const float *src = p.spart + (((size_t)(rg0 + r) * tiles + t) * kWave + (u & 63)) * 4;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            z[i][c] = 16 * r < m ? *reinterpret_cast<const f32x4 *>(src + c * plane) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
    if constexpr (ROWSCALE) {  // the row factors the split launch computed (row_factor_reduce's values)
        if (tid < ROWS) s_inv[tid] = p.sinv[row0 + tid];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int u = tid + i * W * kWave, blk = u >> 6, l = u & 63;
        const int r = blk / NT, j = blk % NT;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int row = 16 * r + 4 * (l >> 4) + v;
            float x = (z[i][0][v] + z[i][2][v]) + (z[i][1][v] + z[i][3][v]);
            if constexpr (ROWSCALE) x *= s_inv[row];
            s_tile[row * (COLS + 1) + 16 * j + (l & 15)] = x;
        }
    }
    __syncthreads();
    gemm_epilogue<P, NT, RG, EP, W>(p, s_tile, s_red, row0, m, wg, tid, lane, w);
}

// The product through the class-pair split: gemm_split_kernel over row_tiles tiles of 64 rows (from
// row tile p.rt0), then gemm_split_reduce_kernel with NT_E tiles per workgroup. e0 marks the
// product's start, e1 the reduction's end.
template <int NT, int NB, int EP, int NT_E>
static hipError_t launch_split_t(const GemmParams &p, int row_tiles, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    constexpr int ROWS = kMaxRows, COLS = 16 * NT;
    constexpr bool ROWSCALE = EP != E_RESID && EP != E_LOGITS;
    if (!p.spart || (ROWSCALE && !p.sinv) || row_tiles < 1 || (p.rt0 + row_tiles) * ROWS > p.rr.cap ||
        p.lda % 32 != 0 || p.cols % 16 != 0 || p.Ks < 4 || p.kc != 0)
        return hipErrorInvalidValue;
    GemmParams q = p;
    q.n_wg = (p.cols + COLS - 1) / COLS;
    q.row_tiles = row_tiles;
    const size_t lds = (size_t)split_lds_floats<4, NT, NB>() * sizeof(float);
    const dim3 grid((unsigned)((q.n_wg + 1) / 2 * 8 * row_tiles));
    auto split = gemm_split_kernel<NT, NB, EP>;
    if (e0)
        hipExtLaunchKernelGGL(split, grid, dim3(kGemmWaves * kWave), lds, s, e0, nullptr, 0, q);
    else
        hipLaunchKernelGGL(split, grid, dim3(kGemmWaves * kWave), lds, s, q);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    GemmParams r = p;
    r.n_wg = (p.cols + 16 * NT_E - 1) / (16 * NT_E);
    r.row_tiles = row_tiles;
    const size_t lds_r = (size_t)split_reduce_lds_floats<NT_E, EP>() * sizeof(float);
    const dim3 grid_r((unsigned)r.n_wg, (unsigned)r.row_tiles);
    auto red = gemm_split_reduce_kernel<NT_E, EP>;
    if (e1)
        hipExtLaunchKernelGGL(red, grid_r, dim3(kGemmWaves * kWave), lds_r, s, nullptr, e1, 0, r);
    else
        hipLaunchKernelGGL(red, grid_r, dim3(kGemmWaves * kWave), lds_r, s, r);
    return hipGetLastError();
}

template <int NT, int RG, int WM, int EP, int NB>
static hipError_t launch_prompt_dma(const GemmParams &p, int rows, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    constexpr int ROWS = 16 * RG, COLS = 16 * NT;
    const size_t lds = (size_t)prompt_dma_lds_floats<NT, RG, EP, NB>() * sizeof(float);
    if (rows < 1 || rows > p.rr.cap || p.rr.cap % ROWS != 0 || p.lda % 32 != 0 || p.cols % 16 != 0)
        return hipErrorInvalidValue;
    GemmParams q = p;
    q.n_wg = (p.cols + COLS - 1) / COLS;
    q.row_tiles = (rows + ROWS - 1) / ROWS;
    const dim3 grid((unsigned)((q.n_wg + 7) / 8 * 8 * q.row_tiles));  // column groups padded to 8 XCDs
    auto kern = gemm_prompt_dma_kernel<NT, RG, WM, EP, NB>;
    if (e0 || e1)
        hipExtLaunchKernelGGL(kern, grid, dim3(kGemmWaves * kWave), lds, s, e0, e1, 0, q);
    else
        hipLaunchKernelGGL(kern, grid, dim3(kGemmWaves * kWave), lds, s, q);
    return hipGetLastError();
}


template <int NT, int RG, int WM, int NB, int NS>
static hipError_t launch_prompt_ksplit(const GemmParams &p, int rows, hipStream_t s, hipEvent_t e0, hipEvent_t e1);

hipError_t launch_gemm_prompt(GemmKind kind, int rows, const GemmParams &p, hipStream_t s, hipEvent_t e0,
                              hipEvent_t e1) {
    switch (kind) {
    // measured at the LLaMA-2-7B shape, 512 rows, random operands: QKV and gate/up take the LDS-DMA
    // kernel with three buffers (64 x 128 tiles for QKV: 114 us, LDS-staged 64 x 256: 167 us;
    // 64 x 256 for gate/up: 177-199 us, LDS-staged: 245 us). O and down, whose 4096 columns give
    // one 64 x 128 workgroup per CU at 512 rows, take the DMA kernel over fixed K ranges and the
    // reduction: O 64 x 128 tiles and 2 ranges (54.6 us against 56.4 for the LDS-staged kernel;
    // 37.1 against 52.3 at 256 rows), down 128 x 128 tiles and 4 ranges (103.5 against 116.0;
    // 61.9 against 102.4 at 256 rows)
    case GEMM_QKV:
        return launch_prompt_dma<8, 4, 2, E_QKV, 3>(p, rows, s, e0, e1);
    case GEMM_GATE_UP:
        return launch_prompt_dma<16, 4, 2, E_SWIGLU, 3>(p, rows, s, e0, e1);
    case GEMM_O:  // X += O W_o^T
        return launch_prompt_ksplit<8, 4, 2, 3, 2>(p, rows, s, e0, e1);
    case GEMM_DOWN:  // X += H W_d^T
        return launch_prompt_ksplit<8, 8, 2, 3, 4>(p, rows, s, e0, e1);
    default:
        return hipErrorInvalidValue;
    }
}

// Grid: column workgroups (ceil(p.cols / (16 * NT))) x row tiles of 16 * RG rows (from row tile
// p.rt0) x K splits (E_LOGITS with p.kc > 0).
template <Prec P, int NT, int RG, int EP, int D = kGemmDepth, int W = kGemmWaves>
static hipError_t launch_gemm_t(const GemmParams &p, int row_tiles, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    constexpr int ROWS = 16 * RG, COLS = 16 * NT;
    static_assert(W * NT * 256 >= ROWS * COLS, "E_RESID reuses the reduction buffer");
    const size_t lds = (size_t)tile_lds_floats<NT, RG, W>() * sizeof(float);
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

// The down product's epilogue: the K-split partial products of kDownSplits workgroups per
// column group summed in a fixed tree, (p0 + p1) + (p2 + p3) (splits past the last are absent
// terms), then X += Y, the next RMSNorm operand X (.) gain (one operand vector per thread) and
// the per-16-column sums of squares: each thread sums its VEC columns in order, the threads of
// a 16-column tile then add their sums in order. Rows past the iteration's rows (device row
// table) exit.
constexpr int kReduceThreads = 64;  // one wave per workgroup: the reduction is latency-bound

template <Prec P>
__global__ __launch_bounds__(kReduceThreads) void down_reduce_kernel(GemmParams p, int nsplit, size_t zstride, int rows_launch) {
    using PT = PrecT<P>;
    using T = typename PT::T;
    constexpr int VEC = PT::VEC, G = 16 / VEC;  // columns per thread, threads per 16-column tile
    const int groups = p.cols / VEC;
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int row = (int)(i / groups), g = (int)(i % groups);  // G consecutive threads share a tile
    const bool live = row < rows_launch && row < p.rr.tab->R;
    float ss = 0.0f;
    if (live) {
        const int c0 = g * VEC;
        const size_t o = (size_t)row * p.ldx + c0;
        float y[VEC], x[VEC];
#pragma unroll
        for (int h = 0; h < VEC / 4; ++h) {
            f32x4 q[kDownSplits];
#pragma unroll
            for (int z = 0; z < kDownSplits; ++z)
                q[z] = z < nsplit ? *reinterpret_cast<const f32x4 *>(p.part + z * zstride + o + 4 * h)
                                  : f32x4{0.f, 0.f, 0.f, 0.f};
            const f32x4 xv = *reinterpret_cast<const f32x4 *>(p.Xout + o + 4 * h);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                y[4 * h + e] = (q[0][e] + q[1][e]) + (q[2][e] + q[3][e]);
                x[4 * h + e] = xv[e] + y[4 * h + e];
            }
        }
        alignas(16) T hi[VEC], lo[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            ss += x[e] * x[e];
            const float a = x[e] * p.gain[c0 + e];
            if constexpr (P == Prec::BF16) {
                hi[e] = f2bf(a);
                lo[e] = f2bf(a - bf2f(hi[e]));
            } else {
                hi[e] = a;
            }
        }
#pragma unroll
        for (int h = 0; h < VEC / 4; ++h)
            *reinterpret_cast<f32x4 *>(p.Xout + o + 4 * h) = f32x4{x[4 * h], x[4 * h + 1], x[4 * h + 2], x[4 * h + 3]};
        T *an = reinterpret_cast<T *>(p.An);
        const size_t ai = act_idx<P>(row, c0, p.ldx);  // VEC consecutive columns: one operand vector
        *reinterpret_cast<u32x4 *>(an + ai) = *reinterpret_cast<const u32x4 *>(hi);
        if constexpr (P == Prec::BF16)
            *reinterpret_cast<u32x4 *>(an + act_plane(p.rr.cap, p.ldx) + ai) = *reinterpret_cast<const u32x4 *>(lo);
    }
    // the tile's G partial sums in order (G consecutive lanes; every lane takes part)
    float tot = 0.0f;
    const int base = (threadIdx.x & 63) & ~(G - 1);
#pragma unroll
    for (int k = 0; k < G; ++k) tot += __shfl(ss, base + k);
    if (live && g % G == 0) p.ssq_out[(size_t)row * p.T + g / G] = tot;
}

// A prompt product with the residual epilogue as NS K ranges through the LDS-DMA kernel (fp32
// partial planes in p.part), then down_reduce_kernel (partials summed in range order, residual,
// next RMSNorm operand and its sums of squares).
template <int NT, int RG, int WM, int NB, int NS>
static hipError_t launch_prompt_ksplit(const GemmParams &p, int rows, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    static_assert(NS >= 1 && NS <= kDownSplits, "down_reduce_kernel sums up to kDownSplits partials");
    constexpr int ROWS = 16 * RG, COLS = 16 * NT;
    if (!p.part || rows < 1 || rows > p.rr.cap || p.rr.cap % ROWS != 0 || p.lda % 32 != 0 || p.cols % 16 != 0 ||
        p.ldx < p.cols || p.Ks < NS)
        return hipErrorInvalidValue;
    GemmParams q = p;
    q.kc = (p.Ks + NS - 1) / NS;
    q.Zout = p.part;
    q.ldz = p.ldx;
    q.V = p.cols;
    q.zstride = (size_t)p.rr.cap * p.ldx;
    q.n_wg = (p.cols + COLS - 1) / COLS;
    q.row_tiles = (rows + ROWS - 1) / ROWS;
    const int nsplit = (p.Ks + q.kc - 1) / q.kc;
    const size_t lds = (size_t)prompt_dma_lds_floats<NT, RG, E_LOGITS, NB>() * sizeof(float);
    const dim3 grid((unsigned)((q.n_wg + 7) / 8 * 8 * q.row_tiles), (unsigned)nsplit);
    auto kern = gemm_prompt_dma_kernel<NT, RG, WM, E_LOGITS, NB>;
    if (e0)
        hipExtLaunchKernelGGL(kern, grid, dim3(kGemmWaves * kWave), lds, s, e0, nullptr, 0, q);
    else
        hipLaunchKernelGGL(kern, grid, dim3(kGemmWaves * kWave), lds, s, q);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    const int rows_launch = q.row_tiles * ROWS;
    const size_t n = (size_t)rows_launch * (p.cols / PrecT<Prec::BF16>::VEC);
    const dim3 grid_r((unsigned)((n + kReduceThreads - 1) / kReduceThreads));
    if (e1)
        hipExtLaunchKernelGGL(down_reduce_kernel<Prec::BF16>, grid_r, dim3(kReduceThreads), 0, s, nullptr, e1, 0, p,
                              nsplit, q.zstride, rows_launch);
    else
        hipLaunchKernelGGL(down_reduce_kernel<Prec::BF16>, grid_r, dim3(kReduceThreads), 0, s, p, nsplit, q.zstride,
                           rows_launch);
    return hipGetLastError();
}

// The down product: K split over kDownSplits ranges (fp32 partials in p.part, 64-column
// workgroups, D k-steps in flight), then down_reduce_kernel. e0 marks the product's start, e1
// the reduction's end.
// ROWK: the split products through the row-tiled kernel (bf16, several row tiles; the same values
// as gemm_kernel's).
template <Prec P, int RG, int D, bool ROWK = false>
static hipError_t launch_down(const GemmParams &p, int row_tiles, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    static_assert(kDownSplits == 4, "down_reduce_kernel sums four partials");
    if (!p.part || p.rt0 != 0 || p.cols % 16 != 0 || p.ldx < p.cols) return hipErrorInvalidValue;
    GemmParams q = p;
    q.kc = (p.Ks + kDownSplits - 1) / kDownSplits;
    q.Zout = p.part;
    q.ldz = p.ldx;
    q.V = p.cols;
    q.zstride = (size_t)p.rr.cap * p.ldx;
    hipError_t err;
    if constexpr (ROWK)
        err = launch_rows_t<kRowsNtDown, E_LOGITS, kRowsNbDown, kLmTiles, D>(q, row_tiles, s, e0, nullptr);
    else
        err = launch_gemm_t<P, kLmTiles, RG, E_LOGITS, D>(q, row_tiles, s, e0, nullptr);
    if (err != hipSuccess) return err;
    const int nsplit = (p.Ks + q.kc - 1) / q.kc;
    const int rows_launch = row_tiles * 16 * RG;
    const size_t n = (size_t)rows_launch * (p.cols / PrecT<P>::VEC);
    const dim3 grid((unsigned)((n + kReduceThreads - 1) / kReduceThreads));
    if (e1)
        hipExtLaunchKernelGGL(down_reduce_kernel<P>, grid, dim3(kReduceThreads), 0, s, nullptr, e1, 0, p, nsplit, q.zstride,
                              rows_launch);
    else
        hipLaunchKernelGGL(down_reduce_kernel<P>, grid, dim3(kReduceThreads), 0, s, p, nsplit, q.zstride, rows_launch);
    return hipGetLastError();
}

template <Prec P, int RG>
static hipError_t launch_gemm_rg(GemmKind kind, const GemmParams &p, int row_tiles, hipStream_t s, hipEvent_t e0,
                                 hipEvent_t e1) {
    if (row_tiles > 1 && P == Prec::BF16 && !p.tile_kernel && p.spart && p.Ks >= 4) {
        // More than 64 rows, bf16 (K of at least four k-steps): QKV, gate/up and the LM head
        // through the class-pair K split (the same values)
        if (kind == GEMM_QKV)
            return launch_split_t<kSplitNtQkv, kSplitNbQkv, E_QKV, 4>(p, row_tiles, s, e0, e1);
        if (kind == GEMM_GATE_UP)
            return launch_split_t<kSplitNtGateUp, kSplitNbGateUp, E_SWIGLU, 4>(p, row_tiles, s, e0, e1);
        // the reduction's column groups are the LM head's argmax workgroups (kLmTiles tiles each)
        if (kind == GEMM_LM)
            return launch_split_t<kSplitNtLm, kSplitNbLm, E_ARGMAX, kLmTiles>(p, row_tiles, s, e0, e1);
    }
    if (row_tiles > 1 && P == Prec::BF16 && !p.tile_kernel) {
        // More than 64 rows, bf16: gate/up and the down product take the row-tiled kernel (the
        // same values); at 7B, 96 / 160 / 256 / 512 rows: gate/up 59 / 112 / 115 / 221 us against
        // 77 / 110 / 144 / 278, down (with its reduction) 36 / 62 / 62 / 116 against 46 / 62 / 80 / 143
        if (kind == GEMM_GATE_UP) return launch_rows_t<kRowsNtGateUp, E_SWIGLU, kRowsNbGateUp, 6, 2>(p, row_tiles, s, e0, e1);
        if (kind == GEMM_DOWN) return launch_down<P, RG, 3, true>(p, row_tiles, s, e0, e1);
    }
    if (row_tiles > 1) {
        // More than 64 rows (measured at 160 and 512 rows, 7B): QKV and gate/up take 96-column
        // workgroups (two k-steps in flight), O and down 64-column workgroups (three k-steps in
        // flight). Row tiles past the iteration's rows exit at once, so a batched iteration
        // launched for its largest row count costs what its live rows cost.
        switch (kind) {
        case GEMM_QKV:
            return launch_gemm_t<P, 6, RG, E_QKV, 2>(p, row_tiles, s, e0, e1);
        case GEMM_O:
            return launch_gemm_t<P, 4, RG, E_RESID, 3>(p, row_tiles, s, e0, e1);
        case GEMM_DOWN:
            return launch_down<P, RG, 3>(p, row_tiles, s, e0, e1);
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
        return launch_gemm_t<P, kNtResid, RG, E_RESID>(p, row_tiles, s, e0, e1);
    case GEMM_DOWN:
        return launch_down<P, RG, kGemmDepth>(p, row_tiles, s, e0, e1);
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

}  // namespace cllm
