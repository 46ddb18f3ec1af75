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
    // The rows' queries (PLANES x NKK vectors per lane) are loaded once per workgroup, one block
    // per wave, and shared through LDS; the first chunk's loads are issued meanwhile.
    constexpr int NQ = PT::PLANES * NKK;
    static_assert(NQ <= W, "one query block per wave");
    __shared__ u32x4 s_q[NQ][kWave];
    u32x4 qblk = u32x4{0u, 0u, 0u, 0u};
    if (w < NQ) {
        const int pl = w / NKK, kk = w % NKK;
        qblk = *reinterpret_cast<const u32x4 *>(Q + pl * act_plane(p.rr.cap, d) +
                                                act_idx<P>(qld, h * HD + kk * PT::KSTEP + g * PT::VEC, d));
    }
    AttnChunk<P, HD> buf[2];
    attn_load_chunk<P, HD>(buf[0], Kh, Vh, chunk_of(0), dt, lane);
    if (w < NQ) s_q[w][lane] = qblk;
    __syncthreads();
    u32x4 qv[PT::PLANES][NKK];
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
        for (int pl = 0; pl < PT::PLANES; ++pl) qv[pl][kk] = s_q[pl * NKK + kk][lane];

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
// Each (h, c, row) writes a partial (max, sum, unnormalised output). With several waves (bf16),
// the chunk's K and V blocks are brought into LDS once per workgroup (LDS DMA, the blocks dealt
// to the waves in turn) and every wave reads its operands there, instead of each wave loading
// the whole chunk from L2; the operands, and so every value, are the same.
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
    const int lane = threadIdx.x & 63, rg = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    constexpr bool SHARED = P == Prec::BF16 && RG > 1;  // K and V staged in LDS for all waves
    if (!SHARED && rbase + 16 * rg >= m) return;  // this wave's rows are all past the block
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

    // K block (kt, kk): keys key0 + 16kt + lane%16, dims kk*KSTEP + (lane/16)*VEC ..; V^T block
    // (dt, kp) (bf16): row = dim 16*dt + lane%16, K slots = keys 32kp+4g+(0..3), 32kp+16+4g+(0..3);
    // the caches hold exactly these 16 bytes per lane contiguously (one KiB per block).
    auto k_block = [&](int kt, int kk) {
        return reinterpret_cast<const u32x4 *>(Kh + ((size_t)((key0 >> 4) + kt) * NKK + kk) * (kWave * PT::VEC)) + lane;
    };
    auto v_block = [&](int dt, int kp) {
        return reinterpret_cast<const u32x4 *>(Vh + ((size_t)((key0 >> 5) + kp) * NDT + dt) * (kWave * 8)) + lane;
    };
    constexpr int NKB = 4 * NKK, NVB = 2 * NDT;  // K and V blocks of the chunk (bf16)
    __shared__ u32x4 s_kv[SHARED ? NKB + NVB : 1][kWave];
    if constexpr (SHARED) {
        static_assert((NKB + NVB) % RG == 0, "every wave issues the same number of blocks");
#pragma unroll
        for (int j = 0; j < (NKB + NVB) / RG; ++j) {
            const int i = rg + j * RG;
            const u32x4 *src = i < NKB ? k_block(i / NKK, i % NKK) : v_block((i - NKB) >> 1, (i - NKB) & 1);
            __builtin_amdgcn_global_load_lds(static_cast<const void *>(src),
                                             (__attribute__((address_space(3))) void *)(&s_kv[i][0]), 16, 0, 0);
        }
    }
    // Every global load of the workgroup is issued up front: Q rows, the chunk's keys and values.
    // A wave whose rows are all past the block (it only helps stage K and V) loads no queries.
    const bool wave_live = rbase + 16 * rg < m;  // uniform over the wave
    u32x4 qv[PT::PLANES][NKK], kv[4][NKK];
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
        const int dcol = h * HD + kk * PT::KSTEP + g * PT::VEC;
#pragma unroll
        for (int pl = 0; pl < PT::PLANES; ++pl)
            qv[pl][kk] = wave_live ? *reinterpret_cast<const u32x4 *>(Q + pl * act_plane(p.rr.cap, d) + act_idx<P>(qld, dcol, d))
                                   : u32x4{0u, 0u, 0u, 0u};
        if constexpr (!SHARED) {
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) kv[kt][kk] = *k_block(kt, kk);
        }
    }
    u32x4 vv[NDT][2];
    if constexpr (P == Prec::BF16 && !SHARED) {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int kp = 0; kp < 2; ++kp) vv[dt][kp] = *v_block(dt, kp);
    }
    if constexpr (SHARED) {
        wait_vm<0>();        // this wave's blocks (and queries) have landed
        barrier_no_fence();  // every wave's
        if (!wave_live) return;  // this wave's rows are all past the block
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
            for (int kt = 0; kt < 4; ++kt) kv[kt][kk] = s_kv[kt * NKK + kk][lane];
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int kp = 0; kp < 2; ++kp) vv[dt][kp] = s_kv[NKB + 2 * dt + kp][lane];
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
// then sums w_c * O_c in chunk order, and the denominator sum w_c * l_c in chunk order beside
// it (each thread forms the same value; no thread waits for another's). The loads are issued
// in two rounds: the row count and the row's position, then the chunk maxima, sums and the
// first kCombinePre chunks' values together.
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
    if (!has_dim) return;
    float num = 0.0f, den = 0.0f;
#pragma unroll
    for (int c = 0; c < kCombinePre; ++c)
        if (c < nlive) {
            den += s_w[c] * s_l[c];
            num += s_w[c] * pre[c];
        }
    int c = kCombinePre;
    for (; c + 4 <= nlive; c += 4) {
        float o[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) o[u] = p.Opart[(b0 + (size_t)(c + u) * cap) * p.hd + dim];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            den += s_w[c + u] * s_l[c + u];
            num += s_w[c + u] * o[u];
        }
    }
    for (; c < nlive; ++c) {
        den += s_w[c] * s_l[c];
        num += s_w[c] * p.Opart[(b0 + (size_t)c * cap) * p.hd + dim];
    }
    put_act<P>(reinterpret_cast<T *>(p.O), act_plane(cap, p.d), act_idx<P>(row, h * p.hd + dim, p.d), num / den);
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

// State update of one sequence after an iteration whose accepted length a is known (one thread):
// commit (L += a), statistics, pending = pred[a-1] and, in a decode, the next block's size and
// where its tokens come from. The emitted tokens and the next block's tokens are written by the
// caller's threads. A prefill chunk commits all its rows (pred[0] is its last row's argmax).
struct NextBlock {
    int newm;     // rows of the next iteration (0: none)
    int e;        // output position of the next block's first token
    int a, m;     // accepted length, rows of the finished iteration
    int usepred;  // z[j] = pred[a-1+j] where a-1+j < m, else a fresh guess draw
    int draw;     // draw index of fresh guesses
};

__device__ void commit_scalar(Ctl *c, int m, int a, int err, int32_t *mlog, int32_t *rec, NextBlock *nb) {
    nb->newm = 0;
    if (err) {
        c->err |= 1;
        c->done = 1;
        c->m = 0;
        return;
    }
    if (c->mode == MODE_PREFILL) {
        c->L += m;
        c->pending = c->pred[0];
        c->m = 0;
        return;
    }
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
    c->e += a;  // z[0..a) were emitted by the caller's threads
    if (c->e >= c->max_new) {
        c->done = 1;
        c->m = 0;
        return;
    }
    const int e = c->e, n = c->n;
    nb->e = e;
    nb->a = a;
    nb->m = m;
    nb->draw = c->policy == 2 ? c->steps : 0;
    if (c->block_policy == 0) {
        if (e == c->b0 + c->nb) {  // block converged; its last prediction seeds the next block
            c->b0 = e;
            c->nb = (c->max_new - e) < n ? (c->max_new - e) : n;
            c->blocks += 1;
            nb->newm = c->nb;
            nb->usepred = 0;
        } else {  // shrink: the unfixed rest of the block
            nb->newm = c->b0 + c->nb - e;
            nb->usepred = c->policy != 2;
        }
    } else {  // slide: the next min(n, remaining) positions
        nb->newm = (c->max_new - e) < n ? (c->max_new - e) : n;
        nb->usepred = c->policy != 2;
    }
    c->z[0] = c->pending;
    c->m = nb->newm;
}

// One workgroup per batch entry: the final argmax of each of its rows over the LM-head
// workgroups (16 threads per row take strided workgroups, then a 16-way tree; (max, lowest id)
// is exact, so the order is free); the accepted length (a = 1 + the leading k >= 1 with
// z[k] = pred[k-1], from one wave's ballot); the emitted tokens; the state update (one thread);
// the next block's tokens (one thread per position). The sequence's control block is worked on
// in LDS (one parallel copy in, one out), so the state update is not a chain of global-memory
// round trips. A prefill chunk that ends its prompt needs only its last row; one that does not
// (and every chunk of a pass without the LM head) only advances L. With one batch entry the workgroup also
// lays out the next row table.
__global__ __launch_bounds__(1024) void scan_commit_kernel(ScanParams p) {
    const int bi = blockIdx.x;
    const RowTab *tab = p.tab;
    if (bi >= tab->nseq) return;
    const int seq = tab->seq[bi];
    const int m = tab->m[bi], r0 = tab->r0[bi];
    Ctl *gc = p.ctl + seq;
    const int tid = threadIdx.x;
    __shared__ int s_pred[kMaxBlock];
    __shared__ NextBlock s_nb;
    __shared__ int s_a, s_err;
    __shared__ Ctl s_ctl;
    static_assert(sizeof(Ctl) % 4 == 0, "the control block is copied as 32-bit words");
    constexpr int kCtlWords = (int)(sizeof(Ctl) / 4);
    if (m > 0) {
        if (p.advance_only || ((p.advance_mask >> bi) & 1)) {
            if (tid == 0) {
                gc->L += m;
                gc->m = 0;
            }
        } else {
            // the copy into LDS overlaps the argmax loads; the barrier after them publishes it
            for (int i = tid; i < kCtlWords; i += blockDim.x)
                reinterpret_cast<int32_t *>(&s_ctl)[i] = reinterpret_cast<const int32_t *>(gc)[i];
            Ctl *c = &s_ctl;
            const bool prefill = gc->mode == MODE_PREFILL;
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
                s_pred[tid] = pr;
                if (rec) {
                    rec[5 + tid] = c->z[tid];
                    rec[5 + kMaxBlock + tid] = pr;
                }
            }
            __syncthreads();
            if (tid < kWave) {  // wave 0: error check, accepted length, emitted tokens
                const bool in = tid < nrows;
                const int zk = in ? c->z[tid] : 0;
                const unsigned long long bad = __ballot(in && s_pred[tid] < 0);
                const unsigned long long miss = __ballot(in && tid >= 1 && zk != s_pred[tid - 1]);
                const int a = miss ? __builtin_ctzll(miss) : nrows;
                if (!bad && !prefill && c->mode == MODE_DECODE && tid < a && p.out) {
                    int32_t *out = p.out + (size_t)seq * p.out_stride;
                    out[c->e + tid] = zk;
                }
                if (tid == 0) {
                    s_a = a;
                    s_err = bad != 0;
                }
            }
            __syncthreads();
            if (tid == 0)
                commit_scalar(c, m, s_a, s_err, p.mlog ? p.mlog + (size_t)seq * p.out_stride : nullptr, rec, &s_nb);
            __syncthreads();
            const int newm = s_nb.newm;
            if (tid >= 1 && tid < newm) {  // the next block's guesses (z[0] = pending, set above)
                const int src = s_nb.a - 1 + tid;
                c->z[tid] = (s_nb.usepred && src < s_nb.m)
                                ? s_pred[src]
                                : draw_guess(c, p.stream ? p.stream + (size_t)seq * p.stream_stride : nullptr,
                                             s_nb.e + tid, s_nb.draw);
            }
            __syncthreads();
            for (int i = tid; i < kCtlWords; i += blockDim.x)
                reinterpret_cast<int32_t *>(gc)[i] = reinterpret_cast<const int32_t *>(&s_ctl)[i];
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
            if ((p.reset_mask >> b) & 1) {
                c->L = 0;
                c->err = 0;
                c->done = 0;
            }
            c->mode = p.mode;
            c->m = p.m[b];
            const size_t zo = p.packed ? (size_t)R : (size_t)b * p.zstride;
            if (p.mode != MODE_PREFILL)
                for (int i = 0; i < p.m[b]; ++i) c->z[i] = p.zin[zo + i];
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
    for (int b = 0; b < p.nseq; ++b) {
        const size_t zo = p.packed ? (size_t)s_r0[b] : (size_t)b * p.zstride;
        for (int i = threadIdx.x; i < p.m[b]; i += blockDim.x)
            p.rows[s_r0[b] + i] = RowInfo{b, s_L[b] + i, p.zin[zo + i], i};
    }
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
