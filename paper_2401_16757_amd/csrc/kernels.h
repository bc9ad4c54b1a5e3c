// kernels.h -- launch interface of the gfx950 kernels used by the swap engine.
//
// All tensors are fp16 (stored as _Float16 on the device) unless noted.
// Activations of image networks are H x W x Cp (channels innermost, Cp a
// multiple of 8); token networks use [T][C].  Weights are in the device
// layout written by the planner: one row per output channel, K contiguous.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sn {

// Implicit-GEMM convolution / token GEMM on MFMA.  Output element
// (m = output pixel or token, n = output channel) is
//   sum_k A[m][k] * W[n][k]  with k = (r, s, ci) over the kh x kw x Cin_p window,
// plus bias, plus residual, then ReLU, rounded once to fp16.
struct ConvArgs {
    const void *x;      // input activation, H x W x Cin_p
    const void *w;      // piece weights, [N rows][K] (rows interleaved gate/up for SwiGLU)
    const void *bias;   // piece bias [N] or null
    const void *res;    // residual activation (same layout as y) or null
    void *y;            // output activation base (channel stride ldy)
    int H, W, Cin_p;
    int Ho, Wo;
    int kh, kw, stride, pad, dil;
    int K;              // kh * kw * Cin_p
    int M;              // Ho * Wo (or tokens)
    int N;              // weight rows in this piece
    int n0;             // first output channel of the piece (in output units)
    int ldy;            // channel stride of y and res
    int n_zero_end;     // zero output channels [n0 + units, n_zero_end) (padding)
    int relu, swiglu;
    // split-K: blockIdx.y = split s covers k in [s*kps, (s+1)*kps); with
    // ksplit > 1 each block writes its partial sums to ws[s][m][n] (fp32)
    // and a second kernel adds them in split order 0..ksplit-1 and applies
    // the epilogue
    int ksplit, kps;
    float *ws;
    int n_cover;        // columns covered by the tile grid (>= N, includes padding)
};

// How a convolution layer is computed: tile variant and K split, chosen from
// the whole layer's (M, N, K) so that every slab piece of the layer runs the
// same reduction order.
struct ConvPlan {
    int kernel = -1;
    int ksplit = 1;
    int kps = 0;
};

// Matrix-vector product for batch-1 linear layers (HBM-bound):
//   y[n0 + n] = sum_k W[n][k] x[k] (+ b[n]) (+ res[n0 + n]) (ReLU)
// SwiGLU: weight rows come in (gate, up) pairs; output unit j is
//   silu(row 2j . x) * (row 2j+1 . x).
struct GemvArgs {
    const void *x;
    const void *w;
    const void *bias;
    const void *res;
    void *y;
    int rows;           // weight rows in this piece
    int K;              // row length (multiple of 8)
    int n0;             // first output unit of the piece
    int relu, swiglu, out_f32;
    int zero_end;       // if > n0 + units: zero outputs [n0 + units, zero_end)
};

// force > 0 (measurement): use tile variant force - 1 wherever its kind
// (general, 1x1 / token GEMM, taps with Cin_p % 64 == 0) is the layer's.
ConvPlan conv_plan(int M, int N, int K, int cin_p, bool is1x1, bool allow_split, int force = 0);
int64_t conv_workspace_bytes(const ConvPlan &p, int M, int N);
int conv_kernel_count();
const char *conv_kernel_name(int id);
// `mid` (optional) is recorded between a K-split convolution's main kernel
// and its reduction.  With `t0` and `t1` (per-piece timing) the kernels are
// launched with start / stop events taken from their own dispatches: t0 at
// the main kernel's start, `mid` (K split) at its end, t1 at the end of the
// last kernel, so that t0 .. t1 is execution time without event overhead.
hipError_t launch_conv(const ConvPlan &p, ConvArgs a, hipStream_t s, hipEvent_t mid = nullptr,
                       hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr);
hipError_t launch_gemv(const GemvArgs &a, hipStream_t s);

hipError_t launch_maxpool(const void *x, void *y, int H, int W, int Cp, int Ho, int Wo, int k,
                          int stride, int pad, hipStream_t s);
hipError_t launch_gavgpool(const void *x, void *y, int HW, int Cp, hipStream_t s);
hipError_t launch_upsample(const void *x, void *y, int H, int W, int Cp, int scale, hipStream_t s);
hipError_t launch_chw_to_hwc(const void *x, void *y, int C, int H, int W, int Cp, hipStream_t s);
hipError_t launch_hwc_to_chw(const void *x, void *y, int C, int H, int W, int Cp, hipStream_t s);

// Swap-in by the compute units: copy `bytes` (a multiple of 16) from pinned
// host memory mapped into the device address space into device memory.
// Ordering against other streams then uses ordinary stream barriers, with no
// host involvement.
hipError_t launch_swapin(const void *src_host_mapped, void *dst, int64_t bytes, int blocks,
                         hipStream_t s);

// Completion signal: increments *flag (a counter in pinned host memory,
// device-mapped) once all earlier work on the stream has finished.  The host
// polls the counter without any runtime call.
hipError_t launch_signal(unsigned long long *flag, hipStream_t s);
// One lane waits (at most limit_ticks of the 100 MHz real-time counter,
// then sets *err) until *value, the value of a ROCr copy's completion
// signal, has dropped to 0.
hipError_t launch_gate(const int64_t *value, unsigned long long limit_ticks, int *err, hipStream_t s);

hipError_t launch_embed(const int32_t *ids, const void *table, void *y, int T, int d, hipStream_t s);
hipError_t launch_rmsnorm(const void *x, const void *gain, void *y, int T, int d, float eps,
                          hipStream_t s);
// RoPE on q and k of each token, append k, v to the cache at pos0 + t, then
// causal attention of every query over cache positions 0 .. pos0 + t.  `ws`
// (attention_workspace_floats(head_dim) floats, or null) holds per-chunk
// partial results when few tokens are processed (decode): the keys are then
// split over several blocks and merged in a fixed order.
constexpr int kAttnWsRecords = 512;
int64_t attention_workspace_floats(int head_dim);
hipError_t launch_attention(const void *qkv, void *kcache, void *vcache, void *q_scratch,
                            void *out, float *ws, int T, int pos0, int heads, int head_dim,
                            float theta, hipStream_t s);

}  // namespace sn
