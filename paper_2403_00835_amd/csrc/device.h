// Device-side types shared by the kernels and the runtime of libcllm.so (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cllm {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;

constexpr int kWave = 64;
constexpr int kMaxBlock = 64;      // largest Jacobi block (rows per iteration)
constexpr int kMaxRows = 64;       // rows of one GEMM row tile; activation buffers hold a multiple
constexpr int kMaxSeqs = 64;       // sequences of one batched iteration
constexpr int kDefaultPrefillRows = 512;  // prompt rows per prefill pass unless the caller sets it
constexpr int kMaxPrefillRows = kMaxSeqs * kMaxBlock;  // = the largest batched iteration
constexpr int kGemmWaves = 8;      // waves per GEMM workgroup; they split K
constexpr int kAttnChunk = 64;     // keys per attention workgroup, at absolute positions
constexpr int kMaxChunks = 1024;   // attention chunks per sequence: context <= 65536
// Trajectory record of one decode iteration (int32): L before it, output position e of z[0],
// block start b0 (shrink policy; e for the slide policy), rows m, accepted a, z[kMaxBlock],
// pred[kMaxBlock].
constexpr int kTraceStride = 5 + 2 * kMaxBlock;
constexpr int kTileBytes = 1024;   // one packed weight tile: 16 rows x 16 bytes x 4 lane groups

// Precision traits. A "k-step" is the K extent one wave covers with one 16-byte load per lane:
// 4 lane groups x VEC elements. bf16: one 16x16x32 MFMA per k-step; fp32: four 16x16x4 MFMAs.
enum class Prec { BF16 = 1, F32 = 0 };
template <Prec P> struct PrecT;
// PLANES: activation operands of the bf16 products carry their fp32 values as two bf16 planes
// (hi = bf16(x), lo = bf16(x - hi): 16 significant bits); fp32 operands have one plane.
template <> struct PrecT<Prec::BF16> {
    using T = uint16_t;  // bf16 bit pattern
    static constexpr int VEC = 8;
    static constexpr int KSTEP = 32;
    static constexpr int PLANES = 2;
};
template <> struct PrecT<Prec::F32> {
    using T = float;
    static constexpr int VEC = 4;
    static constexpr int KSTEP = 16;
    static constexpr int PLANES = 1;
};

__device__ __forceinline__ uint16_t f2bf(float x) {
    __bf16 h = (__bf16)x;  // gfx950 converts with round-to-nearest-even
    return __builtin_bit_cast(uint16_t, h);
}
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

template <Prec P> __device__ __forceinline__ typename PrecT<P>::T to_elem(float x);
template <> __device__ __forceinline__ uint16_t to_elem<Prec::BF16>(float x) { return f2bf(x); }
template <> __device__ __forceinline__ float to_elem<Prec::F32>(float x) { return x; }
template <Prec P> __device__ __forceinline__ float from_elem(typename PrecT<P>::T x);
template <> __device__ __forceinline__ float from_elem<Prec::BF16>(uint16_t x) { return bf2f(x); }
template <> __device__ __forceinline__ float from_elem<Prec::F32>(float x) { return x; }

// Activation operands (the A side of every product, and the attention queries) are stored in the
// MFMA operand order: for 16-row group rg and k-step s, the 64 lanes' 16-byte vectors are
// contiguous (1 KiB), lane = 16 * (k-group within the k-step) + row % 16. A k-step load is one
// contiguous KiB per row group. Each plane holds `rows` rows (the context's row capacity) of K
// elements; the lo plane of a bf16 operand follows the hi plane.
__host__ __device__ constexpr size_t act_plane(int rows, int K) { return (size_t)rows * (size_t)K; }

template <Prec P>
__device__ __forceinline__ size_t act_idx(int row, int k, int K) {
    constexpr int VEC = PrecT<P>::VEC, KSTEP = PrecT<P>::KSTEP;
    const int s = k / KSTEP, w = k % KSTEP;
    return ((size_t)((row >> 4) * (K / KSTEP) + s) * kWave + (w / VEC) * 16 + (row & 15)) * VEC + (w % VEC);
}

// KV cache layout (per sequence slot, layer and head; ctx_alloc * head_dim elements per head), in
// the attention kernel's MFMA operand order so that each load is one contiguous KiB:
//  K:   [pos/16][head_dim/KSTEP][lane 64][VEC], lane = 16 * (dim % KSTEP / VEC) + pos % 16;
//  V^T: bf16 [pos/32][head_dim/16][lane 64][8], lane = 16 * g + dim % 16 where, for key kw =
//       pos % 32, g = (kw % 16) / 4 and the slot is 4 * (kw / 16) + kw % 4 (the probabilities'
//       key order in the score registers); fp32 [pos/16][head_dim/16][lane 64][4],
//       lane = 16 * ((pos % 16) / 4) + dim % 16, slot pos % 4.
template <Prec P>
__device__ __forceinline__ size_t kcache_idx(int pos, int dim, int hd) {
    constexpr int VEC = PrecT<P>::VEC, KSTEP = PrecT<P>::KSTEP;
    return ((size_t)(pos >> 4) * (hd / KSTEP) + dim / KSTEP) * (kWave * VEC) +
           (((dim % KSTEP) / VEC) * 16 + (pos & 15)) * VEC + dim % VEC;
}
template <Prec P>
__device__ __forceinline__ size_t vcache_idx(int pos, int dim, int hd) {
    if constexpr (P == Prec::BF16) {
        const int kw = pos & 31, kq = kw & 15;
        return ((size_t)(pos >> 5) * (hd / 16) + dim / 16) * (kWave * 8) + ((kq >> 2) * 16 + (dim & 15)) * 8 +
               (kw >> 4) * 4 + (kq & 3);
    } else {
        return ((size_t)(pos >> 4) * (hd / 16) + dim / 16) * (kWave * 4) + (((pos & 15) >> 2) * 16 + (dim & 15)) * 4 +
               (pos & 3);
    }
}

// Store x at element i of an activation operand (both planes for bf16).
template <Prec P>
__device__ __forceinline__ void put_act(typename PrecT<P>::T *base, size_t plane, size_t i, float x) {
    if constexpr (P == Prec::BF16) {
        const uint16_t hi = f2bf(x);
        base[i] = hi;
        base[plane + i] = f2bf(x - bf2f(hi));  // x - hi is exact in fp32
    } else {
        base[i] = x;
    }
}

// Makes wave-uniform values available at this point. Kernel prologues list here every
// parameter (and row-table field) their first loads need, so those are requested in one round
// trip; left to itself the compiler requests each one next to its first use, behind the
// branches before it, in several dependent rounds.
template <typename... Ts>
__device__ __forceinline__ void request_together(const Ts &...v) {
    (..., [](const auto &x) { asm volatile("" ::"s"(x)); }(v));
}

// Wait until at most N of this wave's vector memory loads are outstanding (loads retire in
// order, so every older one has landed: for LDS DMA, its bytes are in LDS).
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt holds 6 bits");
    // s_waitcnt with vmcnt = N (bits 3:0 and 15:14) and the other counters at their maxima
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier without the compiler's memory fence (which would wait for every outstanding
// load, DMA included); compiler-only fences keep LDS accesses from moving across it.
__device__ __forceinline__ void barrier_no_fence() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// One k-step of C += A * B on 16x16 tiles. a holds this lane's 16 bytes of the activation row
// (row = lane % 16), b this lane's 16 bytes of the weight row (column = lane % 16); both hold
// the same K indices, so the K-slot assignment inside the instruction does not matter.
template <Prec P> __device__ __forceinline__ f32x4 mfma_kstep(u32x4 a, u32x4 b, f32x4 c);
template <> __device__ __forceinline__ f32x4 mfma_kstep<Prec::BF16>(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
}
template <> __device__ __forceinline__ f32x4 mfma_kstep<Prec::F32>(u32x4 a, u32x4 b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    return c;
}

// Step modes of the shared iteration kernels.
enum StepMode : int32_t {
    MODE_STEP = 0,     // one host-driven iteration: commit a, keep the predictions for the host
    MODE_DECODE = 1,   // device-resident decode: commit, emit, build the next block
    MODE_PREFILL = 2,  // prompt chunk: every row is committed; the last row's argmax is pending
};

// Row table of one iteration. The block rows of every participating sequence are packed in
// batch order: batch entry b (sequence slot seq[b]) owns rows [r0[b], r0[b] + m[b]), at absolute
// positions L[b] .. L[b] + m[b] - 1. Written on the device before each iteration (setup, scan
// and plan kernels); every kernel of the iteration reads it, so one launch sequence serves any
// block sizes.
struct RowTab {
    int32_t R;     // rows of the iteration
    int32_t nseq;  // batch entries
    int32_t pad[2];
    int32_t seq[kMaxSeqs];
    int32_t r0[kMaxSeqs];
    int32_t m[kMaxSeqs];
    int32_t L[kMaxSeqs];
};
struct RowInfo {
    int32_t b;    // batch entry
    int32_t pos;  // absolute position
    int32_t tok;  // token
    int32_t i;    // index within the entry's block
};

// Per-sequence control block, resident on the device. Every kernel of an iteration reads the
// live block length m and the committed length L from here, so one launch sequence (and one
// captured graph) serves every iteration.
struct Ctl {
    int32_t L;         // committed length (cache rows [0, L) are final)
    int32_t m;         // rows of the current iteration (0 = nothing to do)
    int32_t pending;   // known-correct next token (block row 0)
    int32_t mode;      // StepMode
    int32_t e;         // tokens emitted so far in this decode
    int32_t b0, nb;    // first output position and size of the current block (shrink policy)
    int32_t steps, blocks;
    int32_t done;
    int32_t a_last;    // accepted length of the last iteration
    int32_t err;       // bit 0: NaN logit
    int32_t n, max_new;
    int32_t policy, block_policy;
    int32_t seq, stream_len;
    int32_t vocab;
    int32_t rows;      // block rows run by the decode's iterations
    uint64_t seed, thr53;
    int32_t z[kMaxBlock];     // tokens of the current iteration
    int32_t pred[kMaxBlock];  // greedy predictions of the last iteration
    int32_t hist[kMaxBlock + 1];
    int32_t pad1[3];
};

// SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014) and the guess draw of the
// C ABI's guess provider.
__device__ __forceinline__ uint64_t mix64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

}  // namespace cllm
