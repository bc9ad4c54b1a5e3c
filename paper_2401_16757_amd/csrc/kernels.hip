// kernels.hip -- gfx950 (MI355X) kernels of the swap engine.
//
// Compute steps of a block (the per-block execution of the paper's swapping
// cycle, Sec. 3 "Basic Idea"): implicit-GEMM convolution and token GEMM on
// MFMA (v_mfma_f32_32x32x16_f16), a coalesced HBM-bound GEMV for batch-1
// linear layers, pooling, bilinear upsampling, and the decoder's RMSNorm,
// RoPE + attention and embedding gather.
//
// Determinism: every output's reduction order is a function of the layer
// shape only (fixed K order, fixed MFMA instruction, fixed lane-reduction
// tree); splitting a layer by output channels never changes any output bit.
#include "kernels.h"

#include <hip/hip_ext.h>

#include <math.h>

#include <algorithm>
#include <type_traits>
#include <utility>

namespace sn {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Raw buffer loads: a 16-byte load whose byte offset lies past the buffer's
// size returns zeros, so zero padding and ragged edges need no branch.  With
// branch-free loads the compiler counts outstanding loads exactly and the
// prefetched K tiles stay in flight across the loop (a conditional load
// makes it wait for every outstanding load instead).
constexpr unsigned kOobOffset = 0x80000000u;   // buffers are smaller than 2 GiB

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *p, long bytes) {
    // gfx9 descriptor word 3: 32-bit data format, no swizzle, byte-addressed
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ h8 load_h8(__amdgpu_buffer_rsrc_t r, unsigned off) {
    return __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

__device__ __forceinline__ h8 zero_h8() {
    h8 z;
#pragma unroll
    for (int i = 0; i < 8; ++i) z[i] = (_Float16)0.0f;
    return z;
}

__device__ __forceinline__ float silu_f(float v) { return v / (1.0f + expf(-v)); }

// ---------------------------------------------------------------------------
// Implicit-GEMM convolution on MFMA.
//
// Block tile BM (output pixels) x BN (output channels), K tile BK.  The block
// has WM x WN waves; each wave owns a (BM/WM) x (BN/WN) sub-tile made of
// 32 x 32 MFMA tiles.  Operands are staged through LDS (rows padded by 16 B
// against bank conflicts) with the next K tile prefetched into registers
// while the current one is multiplied.
//
// MFMA 32x32x16 lane layout: lane l supplies A[row l%32][k (l/32)*8 .. +7]
// and B[k ...][col l%32]; it receives C[8*(v/4) + 4*(l/32) + v%4][l%32] in
// accumulator register v.
// ---------------------------------------------------------------------------
// Epilogue shared by the MFMA conv kernels: either the K-split partial sums
// (fp32, reduced later in split order) or bias, residual, ReLU / SwiGLU and
// one rounding to fp16, plus zeros in the output's padding channels.
template <int BM, int BN, int WM, int WN>
__device__ __forceinline__ void conv_epilogue(const ConvArgs &a, f16v (&acc)[BM / WM / 32][BN / WN / 32],
                                              int m0, int nb0, int lane, int wm, int wn) {
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    const int lrow = lane & 31;
    if (a.ksplit > 1) {
        // partial sums of this K split; splitk_reduce_kernel adds them
        float *ws = a.ws + (long)blockIdx.y * a.M * a.N;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int n = nb0 + wn * WTN + j * 32 + lrow;
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int m = m0 + wm * WTM + i * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3);
                    if (m < a.M && n < a.N) ws[(long)m * a.N + n] = acc[i][j][v];
                }
            }
        return;
    }

    // Epilogue: bias, residual, ReLU / SwiGLU, one rounding to fp16.
    _Float16 *yg = (_Float16 *)a.y;
    const _Float16 *bg = (const _Float16 *)a.bias;
    const _Float16 *rg = (const _Float16 *)a.res;
    const int units = a.swiglu ? a.N / 2 : a.N;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = nb0 + wn * WTN + j * 32 + lrow;  // weight row (piece-local)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + wm * WTM + i * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3);
                float val = acc[i][j][v];
                if (a.swiglu) {
                    // gate (even row) and up (odd row) sit in adjacent lanes
                    float up = __shfl_xor(val, 1);
                    if ((n & 1) == 0 && m < a.M && n < a.N) {
                        float o = silu_f(val) * up;
                        const long idx = (long)m * a.ldy + a.n0 + (n >> 1);
                        if (rg) o += (float)rg[idx];
                        yg[idx] = (_Float16)o;
                    }
                    continue;
                }
                if (m >= a.M) continue;
                const long idx = (long)m * a.ldy + a.n0 + n;
                if (n < a.N) {
                    if (bg) val += (float)bg[n];
                    if (rg) val += (float)rg[idx];
                    if (a.relu) val = fmaxf(val, 0.0f);
                    yg[idx] = (_Float16)val;
                } else if (a.n0 + n < a.n_zero_end) {
                    yg[idx] = (_Float16)0.0f;
                }
            }
        }
    }
    (void)units;
}


template <int BM, int BN, int BK, int WM, int WN, bool IS1X1>
__global__ __launch_bounds__(WM *WN * 64) void conv_mfma_kernel(ConvArgs a) {
    constexpr int NT = WM * WN * 64;
    constexpr int LDK = BK + 8;            // halves per LDS row
    constexpr int KC = BK / 8;             // 16-byte chunks per row
    constexpr int A_CH = BM * KC / NT;     // A chunks per thread
    constexpr int B_CH = BN * KC / NT;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    static_assert(BM * KC % NT == 0 && BN * KC % NT == 0, "tile/threads mismatch");
    static_assert(TM >= 1 && TN >= 1, "wave tile too small");

    __shared__ _Float16 As[BM * LDK];
    __shared__ _Float16 Bs[BN * LDK];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;

    // Tile coordinates; blockIdx.x walks N tiles fastest so that consecutive
    // blocks share the same activation rows.
    const int n_tiles = (a.n_cover + BN - 1) / BN;
    const int tile_m = blockIdx.x / n_tiles;
    const int tile_n = blockIdx.x % n_tiles;
    const int m0 = tile_m * BM, nb0 = tile_n * BN;

    const int kc = tid % KC;               // same K chunk for all of this thread's rows
    const int row_base = tid / KC;
    constexpr int ROW_STEP = NT / KC;

    const _Float16 *xg = (const _Float16 *)a.x;
    const _Float16 *wg = (const _Float16 *)a.w;

    // Per-row input origin for the A gather.
    int a_iy0[A_CH], a_ix0[A_CH];
    bool a_ok[A_CH];
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
        int m = m0 + row_base + i * ROW_STEP;
        a_ok[i] = m < a.M;
        int oy = a_ok[i] ? m / a.Wo : 0;
        int ox = a_ok[i] ? m - oy * a.Wo : 0;
        a_iy0[i] = oy * a.stride - a.pad;
        a_ix0[i] = ox * a.stride - a.pad;
    }

    h8 ra[A_CH], rb[B_CH];
    auto load_tile = [&](int k0) {
        int k = k0 + kc * 8;
        bool kok = k < a.K;
        int r = 0, s = 0, ci = k;
        if (!IS1X1 && kok) {
            int rs = k / a.Cin_p;
            ci = k - rs * a.Cin_p;
            r = rs / a.kw;
            s = rs - r * a.kw;
        }
#pragma unroll
        for (int i = 0; i < A_CH; ++i) {
            int iy = a_iy0[i] + r * a.dil;
            int ix = a_ix0[i] + s * a.dil;
            bool ok = kok && a_ok[i] && (IS1X1 || (iy >= 0 && iy < a.H && ix >= 0 && ix < a.W));
            ra[i] = ok ? *(const h8 *)(xg + ((long)iy * a.W + ix) * a.Cin_p + ci) : zero_h8();
        }
#pragma unroll
        for (int i = 0; i < B_CH; ++i) {
            int n = nb0 + row_base + i * ROW_STEP;
            bool ok = kok && n < a.N;
            rb[i] = ok ? *(const h8 *)(wg + (long)n * a.K + k) : zero_h8();
        }
    };
    auto store_tile = [&]() {
#pragma unroll
        for (int i = 0; i < A_CH; ++i)
            *(h8 *)(As + (row_base + i * ROW_STEP) * LDK + kc * 8) = ra[i];
#pragma unroll
        for (int i = 0; i < B_CH; ++i)
            *(h8 *)(Bs + (row_base + i * ROW_STEP) * LDK + kc * 8) = rb[i];
    };

    f16v acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    const int lrow = lane & 31;
    const int lk = (lane >> 5) * 8;

    const int kbeg = blockIdx.y * a.kps;
    const int kend = min(a.K, kbeg + a.kps);
    load_tile(kbeg);
    for (int k0 = kbeg; k0 < kend; k0 += BK) {
        __syncthreads();
        store_tile();
        __syncthreads();
        if (k0 + BK < kend) load_tile(k0 + BK);
#pragma unroll
        for (int kk = 0; kk < BK; kk += 16) {
            h8 fa[TM], fb[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                fa[i] = *(const h8 *)(As + (wm * WTM + i * 32 + lrow) * LDK + kk + lk);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                fb[j] = *(const h8 *)(Bs + (wn * WTN + j * 32 + lrow) * LDK + kk + lk);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[i], fb[j], acc[i][j],
                                                                        0, 0, 0);
        }
    }

    conv_epilogue<BM, BN, WM, WN>(a, acc, m0, nb0, lane, wm, wn);
}


// ---------------------------------------------------------------------------
// Multi-stage implicit GEMM with direct global -> LDS loads (gfx950
// buffer_load ... lds, 16 bytes per lane).
//
// Block tile BM x BN, K tile 64, 4 waves in a 2 x 2 grid, S LDS stages: the
// loads of K tile t + S - 1 are in flight while tile t is multiplied, with no
// register staging and one barrier per K tile.  A load instruction of a wave
// fills 8 consecutive LDS rows of 128 bytes, 16 bytes per lane; the lanes
// pick their chunks so that chunk c of row r sits at position c ^ ((r/2) % 8)
// and the MFMA operand reads (16 rows per LDS cycle) hit all 64 banks.  Zero padding and ragged edges are buffer reads past
// the end (zeros).  Each stage is its own LDS variable, which lets the
// compiler track the outstanding LDS loads per stage; the waits before each
// barrier are explicit.
//
// The fp32 tile is finished through LDS 32 rows at a time: every thread
// completes eight consecutive channels of one output pixel with 16-byte
// accesses.  Blocks are renumbered so that each XCD (blocks are dealt to the
// 8 XCDs round-robin) works on a contiguous range of tiles and the operand
// panels they share stay in that XCD's L2.
// ---------------------------------------------------------------------------
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

typedef int i32x4 __attribute__((ext_vector_type(4)));

// f(integral_constant<int, 0>), ..., f(integral_constant<int, N - 1>)
template <class F, int... J>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, J...>) {
    (f(std::integral_constant<int, J>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F &&f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Buffer descriptor (gfx9 layout) of `bytes` bytes at p, in scalar registers.
__device__ __forceinline__ i32x4 make_srd(const void *p, long bytes) {
    const unsigned long long ad = (unsigned long long)p;
    i32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane((int)(unsigned)ad);
    r[1] = __builtin_amdgcn_readfirstlane((int)((ad >> 32) & 0xffffu));   // stride 0
    r[2] = __builtin_amdgcn_readfirstlane((int)bytes);                     // num_records
    r[3] = 0x00020000;                                                     // 32-bit data format
    return r;
}

// LDS address (byte offset in the workgroup's LDS) of a __shared__ pointer.
__device__ __forceinline__ unsigned lds_addr(const void *p) {
    return (unsigned)(size_t)(const __attribute__((address_space(3))) void *)p;
}

// Direct load to LDS: lane l reads 16 bytes at byte offset voff of the
// buffer (zeros past its end) and they land at LDS address lds_base + 16 * l.
// Written as inline assembly so that the compiler neither reorders it against
// LDS reads nor adds waits of its own; completion is counted by vmcnt and
// the callers wait explicitly.  M0 (the LDS base) is saved and restored; one
// wait state separates the M0 write from its use.
__device__ __forceinline__ void dma16_to_lds(i32x4 srd, unsigned lds_base, unsigned voff) {
    // both are wave-uniform by construction; this keeps them in scalar registers
    lds_base = __builtin_amdgcn_readfirstlane(lds_base);
#pragma unroll
    for (int c = 0; c < 4; ++c) srd[c] = __builtin_amdgcn_readfirstlane(srd[c]);
    unsigned saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %2, %3, 0 offen lds\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds_base), "v"(voff), "s"(srd)
        : "memory");
}

// Bias and residual of eight consecutive output channels n .. n+7 of output
// pixel m, loaded ahead of the epilogue (`ok`: the 16-byte path of finish8
// applies, and the values are in `b` / `r`).
struct Pre8 {
    h8 b, r;
    bool ok;
};

__device__ __forceinline__ void prefetch8(const ConvArgs &a, int m, int n, Pre8 &p) {
    p.ok = a.ksplit == 1 && !a.swiglu && m < a.M && (a.n0 % 8) == 0 && n + 8 <= a.N;
    p.b = zero_h8();
    p.r = zero_h8();
    if (!p.ok) return;
    if (a.bias) p.b = *(const h8 *)((const _Float16 *)a.bias + n);
    if (a.res) p.r = *(const h8 *)((const _Float16 *)a.res + (long)m * a.ldy + a.n0 + n);
}

// Bias, residual, ReLU or SwiGLU and the fp16 rounding of eight consecutive
// weight rows n .. n+7 of output pixel m (or their fp32 K-split partials);
// `pre` (optional) holds bias and residual already loaded by prefetch8.
__device__ __forceinline__ void finish8(const ConvArgs &a, int m, int n, float (&v)[8],
                                        const Pre8 *pre = nullptr) {
    if (a.ksplit > 1) {
        float *ws = a.ws + ((long)blockIdx.y * a.M + m) * a.N;
        if (n + 8 <= a.N && (a.N % 4) == 0) {
            *(f4 *)(ws + n) = f4{v[0], v[1], v[2], v[3]};
            *(f4 *)(ws + n + 4) = f4{v[4], v[5], v[6], v[7]};
        } else {
            for (int e = 0; e < 8; ++e)
                if (n + e < a.N) ws[n + e] = v[e];
        }
        return;
    }
    _Float16 *yg = (_Float16 *)a.y;
    const _Float16 *bg = (const _Float16 *)a.bias;
    const _Float16 *rg = (const _Float16 *)a.res;
    if (a.swiglu) {
        // rows come in (gate, up) pairs; unit n/2 + e = silu(gate) * up
        const long idx = (long)m * a.ldy + a.n0 + (n >> 1);
        for (int e = 0; e < 4; ++e) {
            if (n + 2 * e + 1 >= a.N) break;
            float o = silu_f(v[2 * e]) * v[2 * e + 1];
            if (rg) o += (float)rg[idx + e];
            yg[idx + e] = (_Float16)o;
        }
        return;
    }
    const long idx = (long)m * a.ldy + a.n0 + n;
    if (pre && pre->ok) {
        h8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            // the same additions, in the same order, as the paths below
            float x = v[e];
            if (a.bias) x += (float)pre->b[e];
            if (a.res) x += (float)pre->r[e];
            o[e] = (_Float16)(a.relu ? fmaxf(x, 0.0f) : x);
        }
        *(h8 *)(yg + idx) = o;
        return;
    }
    if ((a.n0 % 8) == 0 && n + 8 <= a.N) {
        if (bg) {
            h8 b = *(const h8 *)(bg + n);
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] += (float)b[e];
        }
        if (rg) {
            h8 r = *(const h8 *)(rg + idx);
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] += (float)r[e];
        }
        h8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (_Float16)(a.relu ? fmaxf(v[e], 0.0f) : v[e]);
        *(h8 *)(yg + idx) = o;
        return;
    }
    for (int e = 0; e < 8; ++e) {
        const int ne = n + e;
        if (ne < a.N) {
            float x = v[e];
            if (bg) x += (float)bg[ne];
            if (rg) x += (float)rg[idx + e];
            if (a.relu) x = fmaxf(x, 0.0f);
            yg[idx + e] = (_Float16)x;
        } else if (ne < a.n_cover && a.n0 + ne < a.n_zero_end) {
            yg[idx + e] = (_Float16)0.0f;
        }
    }
}

template <int BM, int BN, int S, int MODE, int KG>
__global__ __launch_bounds__(256 * KG) void conv_mfma3_kernel(ConvArgs a) {
    constexpr int NW = 4 * KG, NT = 64 * NW;   // waves, threads
    constexpr int WTM = BM / 2, WTN = BN / 2;   // wave tile (2 x 2 waves per K group)
    constexpr int TM = WTM / 32, TN = WTN / 32;
    constexpr int QA = BM / 8, QB = BN / 8;     // 8-row load groups per K tile
    // Load groups per wave: NA A groups and NB B groups each, or (when the
    // waves outnumber that split) one group per wave, A for the first QA waves.
    constexpr bool kSplit = QA % NW == 0 && QB % NW == 0;
    constexpr int NA = kSplit ? QA / NW : 1, NB = kSplit ? QB / NW : 1;
    constexpr int NI = kSplit ? NA + NB : 1;    // load instructions per wave per K tile
    constexpr int KPG = 4 / KG;                 // 16-wide K steps per group per K tile
    constexpr int STAGE = (BM + BN) * 64;       // halves per stage
    constexpr int LDC = BN + 4;                 // fp32 staging row
    // epilogue rows staged per round: the whole tile when the K groups'
    // fp32 partials of all BM rows fit in the operand stages, else 64 or 32
    constexpr int RR = KG * BM * LDC * 4 <= S * STAGE * 2 ? BM : KG * 64 * LDC * 4 <= S * STAGE * 2 ? 64 : 32;
    constexpr int ROUNDS = BM / RR;
    static_assert(KG == 1 || KG == 2 || KG == 4, "1, 2 or 4 K groups");
    static_assert(kSplit || QA + QB == NW, "load groups per wave");
    static_assert(S >= 3 && S <= 8, "3 to 8 stages");
    static_assert((S - 1) * NI < 64, "vmcnt range");
    static_assert(KG * RR * LDC * 4 <= S * STAGE * 2 && BM % RR == 0 && RR % 32 == 0,
                  "staging tile exceeds LDS");
    // S operand stages; the epilogue reuses the space for the fp32 partials
    __shared__ __attribute__((aligned(16))) _Float16 smem[S * STAGE];
    auto buf = [&](auto J) -> _Float16 * { return smem + (decltype(J)::value % S) * STAGE; };
    float *stc = (float *)smem;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = KG > 1 ? wave >> 2 : 0;     // K group
    const int wm = (wave >> 1) & 1, wn = wave & 1;

    // XCD-contiguous tile numbering.  Tiles are numbered m-major (the tiles
    // of one XCD share input rows) unless the weight rows outnumber the
    // output pixels (late batch-1 layers): then n-major, so that each weight
    // panel is fetched from HBM by one XCD rather than by every XCD that
    // holds one of its output rows.
    const int nb = gridDim.x, bq = nb >> 3, br = nb & 7;
    const int xcd = blockIdx.x & 7;
    const int lb = xcd * bq + min(xcd, br) + (blockIdx.x >> 3);
    const int n_tiles = (a.n_cover + BN - 1) / BN;
    const int m_tiles = (a.M + BM - 1) / BM;
    const bool n_major = a.n_cover > a.M;
    const int m0 = (n_major ? lb % m_tiles : lb / n_tiles) * BM;
    const int nb0 = (n_major ? lb / m_tiles : lb % n_tiles) * BN;

    const i32x4 xr = make_srd(a.x, (long)a.H * a.W * a.Cin_p * 2);
    const i32x4 wr = make_srd(a.w, (long)a.N * a.K * 2);

    // Lane l takes row l / 8 of each 8-row group it loads and the chunk that
    // puts chunk c of LDS row r at position c ^ ((r / 2) % 8), which spreads
    // the 16 rows read in one LDS cycle over all 64 banks.
    const int lr = lane >> 3;
    const bool wave_a = kSplit || wave < QA;    // half mode: this wave loads A
    const int qa0 = kSplit ? wave * NA : wave;  // first A group of this wave
    const int qb0 = kSplit ? wave * NB : wave - QA;
    int a_iy0[NA], a_ix0[NA], a_off[NA], a_ch[NA];
#pragma unroll
    for (int u = 0; u < NA; ++u) {
        const int row = (qa0 + u) * 8 + lr;
        const int ch = (lane & 7) ^ ((row >> 1) & 7);
        const int m = m0 + row;
        const bool ok = wave_a && m < a.M;
        const int oy = ok ? m / a.Wo : 0;
        const int ox = ok ? m - oy * a.Wo : 0;
        a_ch[u] = ch;
        a_iy0[u] = ok ? oy * a.stride - a.pad : -(1 << 20);   // never inside the input
        a_ix0[u] = ox * a.stride - a.pad;
        // byte offset of the row's first tap (may lie before the buffer)
        a_off[u] = ok ? ((a_iy0[u] * a.W + a_ix0[u]) * a.Cin_p + ch * 8) * 2 : (int)kOobOffset;
    }
    int b_ch[NB];
    unsigned b_off[NB];
#pragma unroll
    for (int u = 0; u < NB; ++u) {
        const int row = (qb0 + u) * 8 + lr;
        const int ch = (lane & 7) ^ ((row >> 1) & 7);
        const int n = nb0 + row;
        b_ch[u] = ch;
        b_off[u] = !wave_a || kSplit ? (n < a.N ? (unsigned)((long)n * a.K + ch * 8) * 2u : kOobOffset)
                                     : kOobOffset;
    }

    const int kbeg = blockIdx.y * a.kps;
    const int kend = min(a.K, kbeg + a.kps);
    int tap_r = 0, tap_s = 0, ci0 = kbeg;
    if (MODE == 1) {
        const int rs = kbeg / a.Cin_p;
        ci0 = kbeg - rs * a.Cin_p;
        tap_r = rs / a.kw;
        tap_s = rs - tap_r * a.kw;
    }

    // loads of the K tile at k0 into stage J (past the K range: zeros)
    auto issue = [&](int k0, auto J) {
        const unsigned sb = lds_addr(buf(J));
        auto load_a = [&]() {
            // tap (r, s) and channel block: a uniform shift of every A row's
            // offset; K tiles never straddle taps, so the range test is uniform
            const int dy = tap_r * a.dil, dx = tap_s * a.dil;
            const int shift = MODE == 1 ? ((dy * a.W + dx) * a.Cin_p + ci0) * 2 : k0 * 2;
#pragma unroll
            for (int u = 0; u < NA; ++u) {
                unsigned off;
                if (MODE == 1) {
                    const bool ok = k0 < kend && (unsigned)(a_iy0[u] + dy) < (unsigned)a.H &&
                                    (unsigned)(a_ix0[u] + dx) < (unsigned)a.W;
                    off = ok ? (unsigned)(a_off[u] + shift) : kOobOffset;
                } else {
                    off = k0 + a_ch[u] * 8 < kend ? (unsigned)a_off[u] + (unsigned)shift : kOobOffset;
                }
                dma16_to_lds(xr, sb + (unsigned)((qa0 + u) * 8 * 128), off);
            }
        };
        auto load_b = [&]() {
#pragma unroll
            for (int u = 0; u < NB; ++u)
                dma16_to_lds(wr, sb + (unsigned)((BM + (qb0 + u) * 8) * 128),
                             k0 + b_ch[u] * 8 < kend ? b_off[u] + (unsigned)k0 * 2u : kOobOffset);
        };
        if constexpr (kSplit) {
            load_a();
            load_b();
        } else {
            if (wave_a) load_a();
            else load_b();
        }
        if (MODE == 1) {
            ci0 += 64;
            if (ci0 >= a.Cin_p) {
                ci0 = 0;
                if (++tap_s == a.kw) {
                    tap_s = 0;
                    ++tap_r;
                }
            }
        }
    };

    f16v acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    const int lrow = lane & 31;
    // LDS element offsets of this lane's operand fragments for the group's
    // 16-wide K steps grp * KPG .. grp * KPG + KPG - 1: chunk kk*2 + lane/32
    // of row lane % 32 of each 32-row MFMA tile (tiles start at multiples of
    // 32 rows)
    int a_rd[KPG][TM], b_rd[KPG][TN];
#pragma unroll
    for (int u = 0; u < KPG; ++u) {
        const int kk = grp * KPG + u;
        const int pos = ((kk * 2 + (lane >> 5)) ^ ((lane >> 1) & 7)) * 8;
#pragma unroll
        for (int i = 0; i < TM; ++i) a_rd[u][i] = (wm * WTM + i * 32 + lrow) * 64 + pos;
#pragma unroll
        for (int j = 0; j < TN; ++j) b_rd[u][j] = BM * 64 + (wn * WTN + j * 32 + lrow) * 64 + pos;
    }
    auto compute = [&](auto J) {
        const _Float16 *sb = buf(J);
        h8 fa[KPG][TM], fb[KPG][TN];
#pragma unroll
        for (int u = 0; u < KPG; ++u) {
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[u][i] = *(const h8 *)(sb + a_rd[u][i]);
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[u][j] = *(const h8 *)(sb + b_rd[u][j]);
        }
#pragma unroll
        for (int u = 0; u < KPG; ++u)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[u][i], fb[u][j], acc[i][j],
                                                                        0, 0, 0);
    };

    const int ntiles = (kend - kbeg + 63) / 64;
    static_for<S - 1>([&](auto J) { issue(kbeg + decltype(J)::value * 64, J); });
    // one K tile per step: wait for its loads (every wave), barrier (also
    // frees the stage multiplied in the previous step), refill that stage
    // with the tile S - 1 ahead, multiply
    auto step = [&](int u, auto J) {
        // the memory clobbers keep the previous step's LDS reads above the
        // wait and the barrier
        asm volatile("" ::: "memory");
        wait_vmcnt<(S - 2) * NI>();
        wait_lgkmcnt0();
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        issue(kbeg + (u + S - 1) * 64, std::integral_constant<int, decltype(J)::value + S - 1>{});
        compute(J);
    };
    // whole groups of S tiles in the loop (its only exit is the condition,
    // which keeps the accumulators in place), then the remainder
    int t = 0;
    for (; t + S <= ntiles; t += S)
        static_for<S>([&](auto J) { step(t + decltype(J)::value, J); });
    const int rem = ntiles - t;
    static_for<S - 1>([&](auto J) {
        if (rem > decltype(J)::value) step(t + decltype(J)::value, J);
    });

    // epilogue: RR rows of the tile per round through LDS (one round where
    // the tile fits: two barriers, one item of eight channels per thread);
    // the bias and residual of every round are loaded first, so their memory
    // latency overlaps the last K tiles instead of being paid once per round
    constexpr int ITEMS = RR * BN / 8;
    constexpr int IPT = (ITEMS + NT - 1) / NT;   // items per thread and round
    Pre8 pre[ROUNDS][IPT];
#pragma unroll
    for (int rd = 0; rd < ROUNDS; ++rd)
#pragma unroll
        for (int u = 0; u < IPT; ++u) {
            const int q = tid + u * NT;
            const int r = q / (BN / 8), n = nb0 + (q % (BN / 8)) * 8;
            pre[rd][u].ok = false;
            if (q < ITEMS) prefetch8(a, m0 + rd * RR + r, n, pre[rd][u]);
        }

    // the loads issued past the end of the K range (zeros) have landed and
    // every wave is done with the operand stages before the epilogue reuses
    // them
    wait_vmcnt<0>();

    // the K groups' partial sums are added in group order
#pragma unroll
    for (int rd = 0; rd < ROUNDS; ++rd) {
        __syncthreads();
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int rb = wm * WTM + i * 32;   // first tile row of this 32-row block
            if (rb / RR == rd) {
                float *dst = stc + (grp * RR + rb % RR) * LDC;
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        dst[((v >> 2) * 8 + (lane >> 5) * 4 + (v & 3)) * LDC + wn * WTN + j * 32 + lrow] =
                            acc[i][j][v];
            }
        }
        __syncthreads();
        const int mb = m0 + rd * RR;
#pragma unroll
        for (int u = 0; u < IPT; ++u) {
            const int q = tid + u * NT;
            const int r = q / (BN / 8), nl = (q % (BN / 8)) * 8;
            const int m = mb + r, n = nb0 + nl;
            if (q < ITEMS && m < a.M && n < a.n_cover) {
                float v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = stc[r * LDC + nl + e];
#pragma unroll
                for (int g = 1; g < KG; ++g)
#pragma unroll
                    for (int e = 0; e < 8; ++e) v[e] += stc[(g * RR + r) * LDC + nl + e];
                finish8(a, m, n, v, &pre[rd][u]);
            }
        }
    }
}

struct ConvVariant {
    int bm, bn, bk;
    int kind;   // 0: conv_mfma (any Cin_p), 4: conv_mfma3 1x1 / token GEMM, 5: conv_mfma3 taps
    const char *name;
    void (*fn)(ConvArgs);
    int threads;
};

#define SN_CONV_VARIANT(BM, BN, BK, WM, WN)                                              \
    {BM, BN, BK, 0, "conv_mfma_" #BM "x" #BN "x" #BK "_w" #WM #WN "_gen",                 \
     conv_mfma_kernel<BM, BN, BK, WM, WN, false>, WM * WN * 64}
#define SN_CONV3_PAIR(BM, BN, S, KG)                                                          \
    {BM, BN, 64, 4, "conv3_mfma_" #BM "x" #BN "_s" #S "_g" #KG "_1x1",                        \
     conv_mfma3_kernel<BM, BN, S, 0, KG>, 256 * KG},                                             \
    {BM, BN, 64, 5, "conv3_mfma_" #BM "x" #BN "_s" #S "_g" #KG "_tap",                        \
     conv_mfma3_kernel<BM, BN, S, 1, KG>, 256 * KG}

static const ConvVariant kConvVariants[] = {
    SN_CONV_VARIANT(128, 128, 32, 2, 2), SN_CONV_VARIANT(128, 64, 32, 2, 2),
    SN_CONV_VARIANT(64, 128, 32, 2, 2),  SN_CONV_VARIANT(64, 64, 32, 2, 2),
    SN_CONV3_PAIR(128, 128, 3, 2),       SN_CONV3_PAIR(64, 128, 4, 2),
    SN_CONV3_PAIR(64, 64, 4, 2),
};
static constexpr int kNumConvVariants = sizeof(kConvVariants) / sizeof(kConvVariants[0]);

int conv_kernel_count() { return kNumConvVariants; }
const char *conv_kernel_name(int id) {
    return (id >= 0 && id < kNumConvVariants) ? kConvVariants[id].name : "?";
}

// Sum of the K-split partials in split order 0..ksplit-1, then bias,
// residual, ReLU and the fp16 rounding; also zeroes the output's padding
// channels.  A separate kernel: the kernel boundary orders the partial-sum
// writes of all splits (on any XCD) before these reads.
__global__ void splitk_reduce_kernel(ConvArgs a) {
    // four consecutive channels per thread
    const int nq = (a.n_cover + 3) / 4;
    long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (long)a.M * nq) return;
    const int m = (int)(t / nq), n = (int)(t - (long)m * nq) * 4;
    _Float16 *yg = (_Float16 *)a.y;
    const long idx = (long)m * a.ldy + a.n0 + n;
    const long plane = (long)a.M * a.N;
    const float *p = a.ws + (long)m * a.N + n;
    float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (n + 4 <= a.N && (a.N % 4) == 0) {
        // loads issued eight splits at a time, added strictly in split order
        int s = 0;
        for (; s + 8 <= a.ksplit; s += 8) {
            f4 q[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) q[e] = *(const f4 *)(p + (long)(s + e) * plane);
#pragma unroll
            for (int e = 0; e < 8; ++e)
#pragma unroll
                for (int c = 0; c < 4; ++c) v[c] += q[e][c];
        }
        for (; s < a.ksplit; ++s) {
            f4 q = *(const f4 *)(p + (long)s * plane);
#pragma unroll
            for (int c = 0; c < 4; ++c) v[c] += q[c];
        }
    } else {
        for (int c = 0; c < 4; ++c)
            if (n + c < a.N)
                for (int s = 0; s < a.ksplit; ++s) v[c] += p[(long)s * plane + c];
    }
    for (int c = 0; c < 4; ++c) {
        const int nc = n + c;
        if (nc >= a.N) {
            if (nc < a.n_cover && a.n0 + nc < a.n_zero_end) yg[idx + c] = (_Float16)0.0f;
            continue;
        }
        float x = v[c];
        if (a.bias) x += (float)((const _Float16 *)a.bias)[nc];
        if (a.res) x += (float)((const _Float16 *)a.res)[idx + c];
        if (a.relu) x = fmaxf(x, 0.0f);
        yg[idx + c] = (_Float16)x;
    }
}

static int find_variant(int bm, int bn, int kind) {
    for (int id = 0; id < kNumConvVariants; ++id)
        if (kConvVariants[id].bm == bm && kConvVariants[id].bn == bn && kConvVariants[id].kind == kind)
            return id;
    return -1;
}

// Tile and K split from the whole layer's shape (never from a slab's channel
// range), so that every piece of a layer runs the same reduction order.
// Batch-1 layers have few output tiles: the largest tile that still gives
// (nearly) every CU a block wins; below that, 64 x 64 tiles, and the K range
// is split only for long reductions on tiny grids (the partial sums cost a
// second pass over ksplit x M x N fp32 values).  1x1 convolutions, token
// GEMMs and taps with Cin_p a multiple of 64 use the multi-stage kernel; the
// rest (the first layer, Cin_p < 64) the single-buffered general one.
ConvPlan conv_plan(int M, int N, int K, int cin_p, bool is1x1, bool allow_split, int force) {
    const int target = 256;
    const int kind = is1x1 ? 4 : (cin_p % 64 == 0 ? 5 : 0);
    ConvPlan p;
    p.kps = K;
    if (force > 0 && force <= kNumConvVariants && kConvVariants[force - 1].kind == kind) {
        p.kernel = force - 1;   // measurement: this variant wherever its kind applies
        return p;
    }
    if (kind == 0) {
        static const int tiles[][2] = {{128, 128}, {128, 64}, {64, 128}, {64, 64}};
        for (auto &t : tiles) {
            const long blocks = (long)((M + t[0] - 1) / t[0]) * ((N + t[1] - 1) / t[1]);
            if (blocks >= target - 16) {
                p.kernel = find_variant(t[0], t[1], kind);
                return p;
            }
        }
        p.kernel = find_variant(64, 64, kind);
        return p;
    }
    static const int tiles[][2] = {{128, 128}, {64, 128}};
    for (auto &t : tiles) {
        if ((t[0] > 64 && M <= 64) || (t[1] > 64 && N <= 64)) continue;
        const long blocks = (long)((M + t[0] - 1) / t[0]) * ((N + t[1] - 1) / t[1]);
        if (blocks >= target - 16) {
            p.kernel = find_variant(t[0], t[1], kind);
            return p;
        }
    }
    p.kernel = find_variant(64, 64, kind);
    const long blocks = (long)((M + 63) / 64) * ((N + 63) / 64);
    const int kt = (K + 63) / 64;
    if (allow_split && blocks <= 32 && K >= 2304) {
        const int s = std::min(8, kt / 2);
        const int per = (kt + s - 1) / s;
        p.kps = per * 64;
        p.ksplit = (K + p.kps - 1) / p.kps;
        if (p.ksplit < 2) {
            p.ksplit = 1;
            p.kps = K;
        }
    }
    return p;
}

int64_t conv_workspace_bytes(const ConvPlan &p, int M, int N) {
    return p.ksplit > 1 ? (int64_t)p.ksplit * M * N * 4 : 0;
}


hipError_t launch_conv(const ConvPlan &p, ConvArgs a, hipStream_t s, hipEvent_t mid, hipEvent_t t0,
                       hipEvent_t t1) {
    if (p.kernel < 0 || p.kernel >= kNumConvVariants) return hipErrorInvalidValue;
    const ConvVariant &v = kConvVariants[p.kernel];
    if (a.M <= 0 || a.N <= 0) return hipSuccess;
    a.ksplit = p.ksplit;
    a.kps = p.ksplit > 1 ? p.kps : a.K;
    if (a.ksplit > 1 && (!a.ws || a.swiglu)) return hipErrorInvalidValue;
    // buffer-load offsets are 32-bit (kOobOffset marks "outside")
    if ((long)a.H * a.W * a.Cin_p * 2 >= (long)kOobOffset || (long)a.N * a.K * 2 >= (long)kOobOffset)
        return hipErrorInvalidValue;
    a.n_cover = std::max(a.N, a.n_zero_end - a.n0);
    long blocks = (long)((a.M + v.bm - 1) / v.bm) * ((a.n_cover + v.bn - 1) / v.bn);
    const dim3 grid((unsigned)blocks, (unsigned)a.ksplit);
    const long n = (long)a.M * ((a.n_cover + 3) / 4);
    const dim3 rgrid((unsigned)((n + 255) / 256));
    if (t0 && t1) {
        // timing: events from the kernels' own dispatches
        hipExtLaunchKernelGGL(v.fn, grid, dim3(v.threads), 0, s, t0, a.ksplit == 1 ? t1 : mid, 0, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess || a.ksplit == 1) return e;
        hipExtLaunchKernelGGL(splitk_reduce_kernel, rgrid, dim3(256), 0, s, nullptr, t1, 0, a);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(v.fn, grid, dim3(v.threads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.ksplit == 1) return e;
    if (mid && (e = hipEventRecord(mid, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(splitk_reduce_kernel, rgrid, dim3(256), 0, s, a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// GEMV (batch-1 linear), HBM-bound: every weight byte is read once.  Each
// wave owns ROWS consecutive weight rows and walks K in steps of 64 x U
// 16-byte chunks: ROWS x U non-temporal weight loads are issued before any
// of them is used (16 KB in flight per wave), the matching input chunks come
// from L1/L2 (the vector is shared by every wave), products are accumulated
// in fp32 in a fixed order, and a fixed butterfly reduces the 64 lanes.
// ---------------------------------------------------------------------------
template <int ROWS, int U>
__global__ __launch_bounds__(256) void gemv_kernel(GemvArgs a) {
    const int tid = threadIdx.x;
    const int kch = a.K / 8;
    if (blockIdx.x == 0 && a.zero_end > 0) {
        const int first = a.n0 + (a.swiglu ? a.rows / 2 : a.rows);
        for (int n = first + tid; n < a.zero_end; n += 256) {
            if (a.out_f32) ((float *)a.y)[n] = 0.0f;
            else ((_Float16 *)a.y)[n] = (_Float16)0.0f;
        }
    }
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int row0 = (blockIdx.x * 4 + wave) * ROWS;
    if (row0 >= a.rows) return;
    const h8 *xg = (const h8 *)a.x;
    const h8 *wrow[ROWS];
#pragma unroll
    for (int r = 0; r < ROWS; ++r)
        wrow[r] = (const h8 *)a.w + (long)min(row0 + r, a.rows - 1) * kch;   // clamped: never out of range

    float acc[ROWS];
#pragma unroll
    for (int r = 0; r < ROWS; ++r) acc[r] = 0.0f;

    int c = lane;
    for (; c + 64 * (U - 1) < kch; c += 64 * U) {
        h8 wv[ROWS][U], xv[U];
#pragma unroll
        for (int r = 0; r < ROWS; ++r)
#pragma unroll
            for (int u = 0; u < U; ++u) wv[r][u] = __builtin_nontemporal_load(wrow[r] + c + 64 * u);
#pragma unroll
        for (int u = 0; u < U; ++u) xv[u] = xg[c + 64 * u];
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
            float sacc = acc[r];
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int i = 0; i < 8; ++i) sacc = fmaf((float)wv[r][u][i], (float)xv[u][i], sacc);
            acc[r] = sacc;
        }
    }
    for (; c < kch; c += 64) {
        const h8 xv = xg[c];
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
            const h8 wv = __builtin_nontemporal_load(wrow[r] + c);
            float sacc = acc[r];
#pragma unroll
            for (int i = 0; i < 8; ++i) sacc = fmaf((float)wv[i], (float)xv[i], sacc);
            acc[r] = sacc;
        }
    }
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
        float v = acc[r];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
        acc[r] = v;
    }
    if (lane != 0) return;
    const _Float16 *bg = (const _Float16 *)a.bias;
    const _Float16 *rg = (const _Float16 *)a.res;
    if (a.swiglu) {
#pragma unroll
        for (int r = 0; r + 1 < ROWS; r += 2) {
            int row = row0 + r;
            if (row + 1 >= a.rows) break;
            int n = a.n0 + (row >> 1);
            float o = silu_f(acc[r]) * acc[r + 1];
            if (rg) o += (float)rg[n];
            if (a.out_f32) ((float *)a.y)[n] = o;
            else ((_Float16 *)a.y)[n] = (_Float16)o;
        }
        return;
    }
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
        int row = row0 + r;
        if (row >= a.rows) break;
        int n = a.n0 + row;
        float o = acc[r];
        if (bg) o += (float)bg[row];
        if (rg) o += (float)rg[n];
        if (a.relu) o = fmaxf(o, 0.0f);
        if (a.out_f32) ((float *)a.y)[n] = o;
        else ((_Float16 *)a.y)[n] = (_Float16)o;
    }
}

hipError_t launch_gemv(const GemvArgs &a, hipStream_t s) {
    if (a.rows <= 0) return hipSuccess;
    if (a.K % 8) return hipErrorInvalidValue;
    constexpr int ROWS = 4;   // even, so SwiGLU pairs stay in one wave
    constexpr int U = 4;
    unsigned blocks = (unsigned)((a.rows + 4 * ROWS - 1) / (4 * ROWS));
    hipLaunchKernelGGL((gemv_kernel<ROWS, U>), dim3(blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Pooling, upsampling and layout conversion (memory-bound, 8 channels per
// thread with 16-byte accesses).
// ---------------------------------------------------------------------------
__global__ void maxpool_kernel(const _Float16 *x, _Float16 *y, int H, int W, int Cp, int Ho,
                               int Wo, int k, int stride, int pad) {
    const int cg = Cp / 8;
    long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (long)Ho * Wo * cg) return;
    int c8 = (int)(t % cg);
    long p = t / cg;
    int ox = (int)(p % Wo), oy = (int)(p / Wo);
    float m[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) m[i] = -INFINITY;
    for (int r = 0; r < k; ++r) {
        int iy = oy * stride - pad + r;
        if (iy < 0 || iy >= H) continue;
        for (int s = 0; s < k; ++s) {
            int ix = ox * stride - pad + s;
            if (ix < 0 || ix >= W) continue;
            h8 v = *(const h8 *)(x + ((long)iy * W + ix) * Cp + c8 * 8);
#pragma unroll
            for (int i = 0; i < 8; ++i) m[i] = fmaxf(m[i], (float)v[i]);
        }
    }
    h8 o;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = (_Float16)m[i];
    *(h8 *)(y + p * Cp + c8 * 8) = o;
}

hipError_t launch_maxpool(const void *x, void *y, int H, int W, int Cp, int Ho, int Wo, int k,
                          int stride, int pad, hipStream_t s) {
    long n = (long)Ho * Wo * (Cp / 8);
    hipLaunchKernelGGL(maxpool_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const _Float16 *)x, (_Float16 *)y, H, W, Cp, Ho, Wo, k, stride, pad);
    return hipGetLastError();
}

// Mean over H*W per channel: one thread per channel, pixels summed in order.
// Mean over H x W per channel.  A block is 16 groups of 8 channels (16-byte
// loads; consecutive threads read consecutive chunks of one pixel) times 16
// pixel lanes; lane l sums pixels l, l + 16, ... in order, then the 16 lane
// sums are added in lane order.  Cp is a multiple of 8.
__global__ void gavgpool_kernel(const _Float16 *x, _Float16 *y, int HW, int Cp) {
    __shared__ float part[16][16][8];
    const int g = threadIdx.x & 15, pl = threadIdx.x >> 4;
    const int c8 = blockIdx.x * 16 + g;
    const bool ok = c8 * 8 < Cp;
    float acc[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    if (ok)
        for (int p = pl; p < HW; p += 16) {
            const h8 v = *(const h8 *)(x + (long)p * Cp + c8 * 8);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] += (float)v[e];
        }
#pragma unroll
    for (int e = 0; e < 8; ++e) part[pl][g][e] = acc[e];
    __syncthreads();
    if (pl != 0 || !ok) return;
    h8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        float t = part[0][g][e];
        for (int l = 1; l < 16; ++l) t += part[l][g][e];
        o[e] = (_Float16)(t / (float)HW);
    }
    *(h8 *)(y + c8 * 8) = o;
}

hipError_t launch_gavgpool(const void *x, void *y, int HW, int Cp, hipStream_t s) {
    if (Cp % 8) return hipErrorInvalidValue;
    hipLaunchKernelGGL(gavgpool_kernel, dim3((Cp / 8 + 15) / 16), dim3(256), 0, s, (const _Float16 *)x,
                       (_Float16 *)y, HW, Cp);
    return hipGetLastError();
}

// Bilinear, integer factor, half-pixel centres: source = (o + 0.5)/scale - 0.5
// clamped at 0, upper neighbour clamped to the edge.
__global__ void upsample_kernel(const _Float16 *x, _Float16 *y, int H, int W, int Cp, int scale) {
    const int cg = Cp / 8;
    const int Ho = H * scale, Wo = W * scale;
    long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (long)Ho * Wo * cg) return;
    int c8 = (int)(t % cg);
    long p = t / cg;
    int ox = (int)(p % Wo), oy = (int)(p / Wo);
    float inv = 1.0f / (float)scale;
    float sy = fmaxf(((float)oy + 0.5f) * inv - 0.5f, 0.0f);
    float sx = fmaxf(((float)ox + 0.5f) * inv - 0.5f, 0.0f);
    int y0 = min((int)sy, H - 1), x0 = min((int)sx, W - 1);
    int y1 = min(y0 + 1, H - 1), x1 = min(x0 + 1, W - 1);
    float ly = sy - (float)y0, lx = sx - (float)x0;
    h8 a = *(const h8 *)(x + ((long)y0 * W + x0) * Cp + c8 * 8);
    h8 b = *(const h8 *)(x + ((long)y0 * W + x1) * Cp + c8 * 8);
    h8 c = *(const h8 *)(x + ((long)y1 * W + x0) * Cp + c8 * 8);
    h8 d = *(const h8 *)(x + ((long)y1 * W + x1) * Cp + c8 * 8);
    h8 o;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        float top = (float)a[i] * (1.0f - lx) + (float)b[i] * lx;
        float bot = (float)c[i] * (1.0f - lx) + (float)d[i] * lx;
        o[i] = (_Float16)(top * (1.0f - ly) + bot * ly);
    }
    *(h8 *)(y + p * Cp + c8 * 8) = o;
}

hipError_t launch_upsample(const void *x, void *y, int H, int W, int Cp, int scale, hipStream_t s) {
    long n = (long)H * scale * W * scale * (Cp / 8);
    hipLaunchKernelGGL(upsample_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const _Float16 *)x, (_Float16 *)y, H, W, Cp, scale);
    return hipGetLastError();
}

__global__ void chw_to_hwc_kernel(const _Float16 *x, _Float16 *y, int C, int HW, int Cp) {
    long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (long)HW * Cp) return;
    int c = (int)(t % Cp);
    long p = t / Cp;
    y[t] = c < C ? x[(long)c * HW + p] : (_Float16)0.0f;
}

hipError_t launch_chw_to_hwc(const void *x, void *y, int C, int H, int W, int Cp, hipStream_t s) {
    long n = (long)H * W * Cp;
    hipLaunchKernelGGL(chw_to_hwc_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const _Float16 *)x, (_Float16 *)y, C, H * W, Cp);
    return hipGetLastError();
}

__global__ void hwc_to_chw_kernel(const _Float16 *x, _Float16 *y, int C, int HW, int Cp) {
    long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (long)HW * C) return;
    long p = t % HW;
    int c = (int)(t / HW);
    y[t] = x[p * Cp + c];
}

hipError_t launch_hwc_to_chw(const void *x, void *y, int C, int H, int W, int Cp, hipStream_t s) {
    long n = (long)H * W * C;
    hipLaunchKernelGGL(hwc_to_chw_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const _Float16 *)x, (_Float16 *)y, C, H * W, Cp);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Swap-in copy kernel: each thread keeps four 16-byte host reads in flight;
// reads are non-temporal (the image is read once per inference).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void swapin_kernel(const u32x4 *__restrict__ src,
                                                     u32x4 *__restrict__ dst, long n16) {
    const long stride = (long)gridDim.x * 256;
    long i = (long)blockIdx.x * 256 + threadIdx.x;
    for (; i + 3 * stride < n16; i += 4 * stride) {
        u32x4 a = __builtin_nontemporal_load(src + i);
        u32x4 b = __builtin_nontemporal_load(src + i + stride);
        u32x4 c = __builtin_nontemporal_load(src + i + 2 * stride);
        u32x4 d = __builtin_nontemporal_load(src + i + 3 * stride);
        dst[i] = a;
        dst[i + stride] = b;
        dst[i + 2 * stride] = c;
        dst[i + 3 * stride] = d;
    }
    for (; i < n16; i += stride) dst[i] = __builtin_nontemporal_load(src + i);
}

hipError_t launch_swapin(const void *src_host_mapped, void *dst, int64_t bytes, int blocks,
                         hipStream_t s) {
    if (bytes <= 0) return hipSuccess;
    if (bytes % 16) return hipErrorInvalidValue;
    const long n16 = bytes / 16;
    long need = (n16 + 1023) / 1024;   // at least 4 chunks per thread
    unsigned grid = (unsigned)std::max<long>(1, std::min<long>(blocks, need));
    hipLaunchKernelGGL(swapin_kernel, dim3(grid), dim3(256), 0, s, (const u32x4 *)src_host_mapped,
                       (u32x4 *)dst, n16);
    return hipGetLastError();
}

__global__ void signal_kernel(unsigned long long *flag) {
    if (threadIdx.x == 0) *(volatile unsigned long long *)flag = *(volatile unsigned long long *)flag + 1;
}

hipError_t launch_signal(unsigned long long *flag, hipStream_t s) {
    hipLaunchKernelGGL(signal_kernel, dim3(1), dim3(64), 0, s, flag);
    return hipGetLastError();
}

// Gate of a slab whose swap-in runs on the SDMA engine through ROCr: one lane
// polls the copy's completion signal value (1 while the copy runs, 0 once it
// has landed) and returns when it reaches 0, so the kernels queued behind it
// on the stream start after the copy.  The wait is bounded: after
// `limit_ticks` of the 100 MHz real-time counter the lane sets *err and
// returns.
__global__ void gate_kernel(const int64_t *value, unsigned long long limit_ticks, int *err) {
    if (threadIdx.x != 0) return;
    const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
    while (__hip_atomic_load(value, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM) > 0) {
        if (__builtin_amdgcn_s_memrealtime() - t0 > limit_ticks) {
            __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
            return;
        }
        __builtin_amdgcn_s_sleep(2);
    }
}

hipError_t launch_gate(const int64_t *value, unsigned long long limit_ticks, int *err, hipStream_t s) {
    hipLaunchKernelGGL(gate_kernel, dim3(1), dim3(64), 0, s, value, limit_ticks, err);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Decoder kernels.
// ---------------------------------------------------------------------------

// Embedding rows gathered straight from the pinned host table (mapped into
// the device address space): only the rows of the given ids cross the link.
__global__ void embed_kernel(const int32_t *ids, const _Float16 *table, _Float16 *y, int d) {
    int t = blockIdx.x;
    long row = ids[t];
    const h8 *src = (const h8 *)(table + row * d);
    h8 *dst = (h8 *)(y + (long)t * d);
    for (int c = threadIdx.x; c < d / 8; c += blockDim.x) dst[c] = src[c];
}

hipError_t launch_embed(const int32_t *ids, const void *table, void *y, int T, int d, hipStream_t s) {
    hipLaunchKernelGGL(embed_kernel, dim3(T), dim3(256), 0, s, ids, (const _Float16 *)table,
                       (_Float16 *)y, d);
    return hipGetLastError();
}

// Block-wide fixed-order sum (256 threads).
__device__ float block_sum_256(float v, float *red) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    const int wave = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[wave] = v;
    __syncthreads();
    return (red[0] + red[1]) + (red[2] + red[3]);
}

// One block per token; 8 channels per thread with 16-byte accesses when d is
// a multiple of 8.  Sum of squares in a fixed order (per-thread strided
// partials, then the block reduction).
__global__ __launch_bounds__(256) void rmsnorm_kernel(const _Float16 *x, const _Float16 *g,
                                                      _Float16 *y, int d, float eps) {
    __shared__ float red[4];
    const _Float16 *xr = x + (long)blockIdx.x * d;
    _Float16 *yr = y + (long)blockIdx.x * d;
    const bool vec = (d % 8) == 0;
    float s = 0.0f;
    if (vec) {
        for (int c = threadIdx.x; c < d / 8; c += 256) {
            const h8 v = *(const h8 *)(xr + 8 * c);
#pragma unroll
            for (int e = 0; e < 8; ++e) s = fmaf((float)v[e], (float)v[e], s);
        }
    } else {
        for (int c = threadIdx.x; c < d; c += 256) {
            float v = (float)xr[c];
            s = fmaf(v, v, s);
        }
    }
    s = block_sum_256(s, red);
    const float scale = 1.0f / sqrtf(s / (float)d + eps);
    if (vec) {
        for (int c = threadIdx.x; c < d / 8; c += 256) {
            const h8 v = *(const h8 *)(xr + 8 * c), gv = *(const h8 *)(g + 8 * c);
            h8 o;
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = (_Float16)((float)v[e] * scale * (float)gv[e]);
            *(h8 *)(yr + 8 * c) = o;
        }
    } else {
        for (int c = threadIdx.x; c < d; c += 256) yr[c] = (_Float16)((float)xr[c] * scale * (float)g[c]);
    }
}

hipError_t launch_rmsnorm(const void *x, const void *gain, void *y, int T, int d, float eps,
                          hipStream_t s) {
    hipLaunchKernelGGL(rmsnorm_kernel, dim3(T), dim3(256), 0, s, (const _Float16 *)x,
                       (const _Float16 *)gain, (_Float16 *)y, d, eps);
    return hipGetLastError();
}

// RoPE (rotate-half) on q and k; q goes to q_scratch (fp32), k and v to the
// cache at position pos0 + t.  One block per token.  The rotation angle of
// pair i at position p is p * theta^(-2i/hd), evaluated once per pair index
// in double precision (shared by all heads), its cosine and sine rounded to
// fp32.
__global__ void rope_append_kernel(const _Float16 *qkv, float *qs, _Float16 *kc, _Float16 *vc,
                                   int pos0, int heads, int hd, float theta) {
    extern __shared__ float cs_sn[];   // [half] cosines, then [half] sines
    const int t = blockIdx.x;
    const int d = heads * hd;
    const int half = hd / 2;
    const _Float16 *row = qkv + (long)t * 3 * d;
    const long pos = pos0 + t;
    for (int i = threadIdx.x; i < half; i += blockDim.x) {
        const double ang = (double)pos * pow((double)theta, -2.0 * (double)i / (double)hd);
        cs_sn[i] = (float)cos(ang);
        cs_sn[half + i] = (float)sin(ang);
    }
    __syncthreads();
    for (int p = threadIdx.x; p < heads * half; p += blockDim.x) {
        const int h = p / half, i = p - h * half;
        const float cs = cs_sn[i], sn = cs_sn[half + i];
        const int a = h * hd + i, b = a + half;
        const float qa = (float)row[a], qb = (float)row[b];
        qs[(long)t * d + a] = qa * cs - qb * sn;
        qs[(long)t * d + b] = qb * cs + qa * sn;
        const float ka = (float)row[d + a], kb = (float)row[d + b];
        kc[pos * d + a] = (_Float16)(ka * cs - kb * sn);
        kc[pos * d + b] = (_Float16)(kb * cs + ka * sn);
        vc[pos * d + a] = row[2 * d + a];
        vc[pos * d + b] = row[2 * d + b];
    }
}

// Causal attention for head_dim a power of two in [8, 512].  A key row
// (head_dim fp16) is read by LPK = head_dim/8 lanes with one 16-byte load
// each, so a block covers 256/LPK keys per step with coalesced loads.
// Scores go to LDS; max and sum are block reductions in a fixed order; for
// P.V every LPK-lane group accumulates its keys (group, group + G, ...) in
// order and the G partial vectors are added in group order.
//   SPLIT = false: one block per (token, head) writes the output.
//   SPLIT = true (few tokens, i.e. decode): the keys of each (token, head)
//   are cut into S consecutive chunks, one block each, which write their
//   partial max, sum and unnormalised output to a workspace;
//   attention_combine_kernel merges the S chunks in order.
// Every result depends on the position only, never on timing.
template <int LPK, bool SPLIT>
__global__ __launch_bounds__(256) void attention_kernel(const float *qs, const _Float16 *kc,
                                                        const _Float16 *vc, _Float16 *out,
                                                        float *ws, int pos0, int heads, int S) {
    constexpr int HD = LPK * 8;
    constexpr int G = 256 / LPK;                    // lane groups (keys per step)
    extern __shared__ float smem[];                 // scores [chunk], then partials [G][HD]
    __shared__ float red[4];
    const int bh = SPLIT ? blockIdx.x / S : blockIdx.x;
    const int split = SPLIT ? blockIdx.x % S : 0;
    const int t = bh / heads, h = bh % heads;
    const int d = heads * HD;
    const int nk = pos0 + t + 1;
    const int chunk = SPLIT ? (pos0 + (int)(gridDim.x / S / heads) + S - 1) / S : nk;   // same for every token
    const int j0 = split * chunk, j1 = min(nk, j0 + chunk);
    float *sc = smem;
    float *part = smem + ((chunk + 3) & ~3);
    const int grp = threadIdx.x / LPK, l = threadIdx.x % LPK;
    const float scale = 1.0f / sqrtf((float)HD);

    float q[8];
    {
        const float *qp = qs + (long)t * d + h * HD + 8 * l;
        const f4 q0 = *(const f4 *)qp, q1 = *(const f4 *)(qp + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            q[e] = q0[e];
            q[4 + e] = q1[e];
        }
    }
    const _Float16 *kb = kc + h * HD + 8 * l;
    const _Float16 *vb = vc + h * HD + 8 * l;
    for (int j = j0 + grp; j < j1; j += G) {
        const h8 k = *(const h8 *)(kb + (long)j * d);
        float s = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) s = fmaf(q[e], (float)k[e], s);
#pragma unroll
        for (int off = LPK / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off);
        if (l == 0) sc[j - j0] = s * scale;
    }
    __syncthreads();
    float m = -INFINITY;
    for (int j = j0 + threadIdx.x; j < j1; j += 256) m = fmaxf(m, sc[j - j0]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    __syncthreads();
    float sum = 0.0f;
    for (int j = j0 + threadIdx.x; j < j1; j += 256) {
        const float e = expf(sc[j - j0] - m);
        sc[j - j0] = e;
        sum += e;
    }
    sum = block_sum_256(sum, red);   // also orders the sc[] writes before the reads below
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = 0.0f;
    for (int j = j0 + grp; j < j1; j += G) {
        const h8 v = *(const h8 *)(vb + (long)j * d);
        const float p = sc[j - j0];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = fmaf(p, (float)v[e], o[e]);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) part[grp * HD + 8 * l + e] = o[e];
    __syncthreads();
    if (SPLIT) {
        // chunk record: [HD] unnormalised output, then max, sum (an empty
        // chunk has max -inf and sum 0 and adds nothing when merged)
        float *rec = ws + (long)blockIdx.x * (HD + 2);
        for (int i = threadIdx.x; i < HD; i += 256) {
            float acc = 0.0f;
            for (int g2 = 0; g2 < G; ++g2) acc += part[g2 * HD + i];
            rec[i] = acc;
        }
        if (threadIdx.x == 0) {
            rec[HD] = j0 < j1 ? m : -INFINITY;
            rec[HD + 1] = sum;
        }
        return;
    }
    const float inv = 1.0f / sum;
    for (int i = threadIdx.x; i < HD; i += 256) {
        float acc = 0.0f;
        for (int g2 = 0; g2 < G; ++g2) acc += part[g2 * HD + i];
        out[(long)t * d + h * HD + i] = (_Float16)(acc * inv);
    }
}

// Merges the S chunk records of each (token, head) in chunk order:
// out = sum_s exp(m_s - M) o_s / sum_s exp(m_s - M) l_s with M = max_s m_s.
__global__ __launch_bounds__(256) void attention_combine_kernel(const float *ws, _Float16 *out,
                                                                int heads, int hd, int S) {
    const int bh = blockIdx.x;
    const int t = bh / heads, h = bh % heads;
    const float *rec = ws + (long)bh * S * (hd + 2);
    float M = -INFINITY;
    for (int s = 0; s < S; ++s) M = fmaxf(M, rec[s * (hd + 2) + hd]);
    float L = 0.0f;
    for (int s = 0; s < S; ++s) {
        const float ms = rec[s * (hd + 2) + hd];
        if (ms != -INFINITY) L += expf(ms - M) * rec[s * (hd + 2) + hd + 1];
    }
    const float inv = 1.0f / L;
    for (int i = threadIdx.x; i < hd; i += 256) {
        float acc = 0.0f;
        for (int s = 0; s < S; ++s) {
            const float ms = rec[s * (hd + 2) + hd];
            if (ms != -INFINITY) acc += expf(ms - M) * rec[s * (hd + 2) + i];
        }
        out[(long)t * heads * hd + h * hd + i] = (_Float16)(acc * inv);
    }
}

int64_t attention_workspace_floats(int head_dim) { return (int64_t)kAttnWsRecords * (head_dim + 2); }

hipError_t launch_attention(const void *qkv, void *kcache, void *vcache, void *q_scratch,
                            void *out, float *ws, int T, int pos0, int heads, int head_dim,
                            float theta, hipStream_t s) {
    if (head_dim % 8 || head_dim < 8 || head_dim > 512 || (head_dim & (head_dim - 1)))
        return hipErrorInvalidValue;   // power of two, 8 .. 512
    hipLaunchKernelGGL(rope_append_kernel, dim3(T), dim3(256), (size_t)head_dim * sizeof(float), s,
                       (const _Float16 *)qkv, (float *)q_scratch, (_Float16 *)kcache,
                       (_Float16 *)vcache, pos0, heads, head_dim, theta);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int lpk = head_dim / 8;
    const int nk_max = pos0 + T;
    // few (token, head) pairs: split the keys so that about 256 blocks run,
    // each over at least 64 keys, within the workspace
    int S = 1;
    if (ws && T * heads < 256) {
        S = std::min(std::min(16, (256 + T * heads - 1) / (T * heads)), (nk_max + 63) / 64);
        while (S > 1 && (int64_t)T * heads * S > kAttnWsRecords) --S;
    }
    const int chunk = S > 1 ? (nk_max + S - 1) / S : nk_max;
    const size_t lds = ((size_t)((chunk + 3) & ~3) + (size_t)(256 / lpk) * head_dim) * sizeof(float);
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3(T * heads * S), dim3(256), lds, s, (const float *)q_scratch,
                           (const _Float16 *)kcache, (const _Float16 *)vcache, (_Float16 *)out, ws,
                           pos0, heads, S);
    };
    if (S > 1) {
        switch (lpk) {
        case 1: go(attention_kernel<1, true>); break;
        case 2: go(attention_kernel<2, true>); break;
        case 4: go(attention_kernel<4, true>); break;
        case 8: go(attention_kernel<8, true>); break;
        case 16: go(attention_kernel<16, true>); break;
        case 32: go(attention_kernel<32, true>); break;
        default: go(attention_kernel<64, true>); break;
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(attention_combine_kernel, dim3(T * heads), dim3(256), 0, s,
                           (const float *)ws, (_Float16 *)out, heads, head_dim, S);
        return hipGetLastError();
    }
    switch (lpk) {
    case 1: go(attention_kernel<1, false>); break;
    case 2: go(attention_kernel<2, false>); break;
    case 4: go(attention_kernel<4, false>); break;
    case 8: go(attention_kernel<8, false>); break;
    case 16: go(attention_kernel<16, false>); break;
    case 32: go(attention_kernel<32, false>); break;
    default: go(attention_kernel<64, false>); break;
    }
    return hipGetLastError();
}

}  // namespace sn
