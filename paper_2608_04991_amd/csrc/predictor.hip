// predictor.hip - gfx950 kernels and C ABI of the decode-phase reference
// predictor: a one-layer causal Transformer over a sequence's earlier
// boundary states with a bounded key-value cache (the paper's subsection
// "Predicted References for Decode", Eq. decode-predictor).  For t >= 2 it
// turns the previous reconstructed state H-hat^{t-1} of every sequence of a
// decode batch into the reference R_pred^t that the codec then encodes
// against.  The contract of each entry point is documented in include/rac.h.
//
// One step (every launch on the caller's stream; B sequences, width d, model
// width m, h heads of 64 channels, SwiGLU width f, window W):
//   h0 = x W_in^T                                     (x = H-hat^{t-1}, bf16)
//   q, k, v = RMSNorm(h0; g1) W_qkv^T, rotary positions on q and k
//   o  = softmax(q k^T / 8) v over the last min(pos + 1, W) inputs
//   h1 = h0 + o W_o^T
//   h2 = h1 + (silu(n2 W_gate^T) * (n2 W_up^T)) W_down^T,  n2 = RMSNorm(h1; g2)
//   R  = x + RMSNorm(h2; g3) W_out^T                  (bf16)
// The products are bf16 x bf16 with fp32 accumulation on the matrix cores
// (v_mfma_f32_16x16x32_bf16); the residual stream h0..h2 is fp32; the
// normalized activations, o, the SwiGLU output and the cached keys and values
// are bf16.
//
// Mapping onto CDNA4.  Decode batches are skinny (B <= 256 rows against
// weight matrices of up to 4096 x 4096), so the products are weight-streaming:
// a workgroup owns 16 output columns and a K range, its four wavefronts split
// that range and sum their accumulators through LDS in a fixed order, and
// long K ranges are split further across workgroups (partials summed, again
// in a fixed order, by the row kernel that follows).  Every weight byte is
// read once per 64 batch rows.
#include <hip/hip_runtime.h>

#include <cmath>
#include <stddef.h>
#include <stdint.h>

#include "rac.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kW = 64;           // wavefront
constexpr int kGemmWaves = 4;
constexpr int kNt = 16;          // output columns per workgroup
constexpr int kRt = 4;           // 16-row tiles per workgroup (64 batch rows)
constexpr int kHd = 64;          // channels per head
constexpr float kEps = 1e-6f;    // RMSNorm

__device__ __forceinline__ float bf(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ uint16_t to_bf(float v) {  // round to nearest even (finite)
    const uint32_t u = __float_as_uint(v);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// ---------------------------------------------------------------------------
// C[b][n] = sum_k A[b][k] W[n][k] over one K range, A bf16 [M][K] row-major,
// W bf16 [N][K] (each output's weights contiguous).  Grid: x = N / 16 column
// tiles, y = K splits, z = 64-row tiles of the batch.  In one MFMA
// (16 x 16 x 32) lane l holds A[l % 16][8 (l / 16) + j] and
// W[n0 + l % 16][8 (l / 16) + j], j < 8, each one 16-byte load, and gets
// C[4 (l / 16) + r][n0 + l % 16], r < 4.
enum Epi { kPartial = 0, kStore = 1, kSwiglu = 2, kResidOut = 3 };

struct Gemm {
    const uint16_t* a;   // [M][K] (not read with NORM)
    const uint16_t* w;   // [N][K]
    int32_t M, N, K, ksplit;   // K range per split
    float* out;          // kPartial: [splits][M][N]; kStore: [M][N]
    uint16_t* out16;     // kSwiglu: [M][N/2]; kResidOut: [M][N]
    const uint16_t* resid;     // kResidOut: bf16 [M][N] added to the product
    // NORM (M <= kFuseRows, one K range, K <= kFuseK): the activations are
    // bf16(h / sqrt(mean(h^2) + eps) * gain), h = nres + sum_s npart[s] added
    // in order, formed by every workgroup in LDS (the norm of the step's row
    // kernel, folded into the product that consumes it)
    const float* nres;      // [M][K], or null
    const float* npart;     // [nsplits][M][K]
    int32_t nsplits;
    const uint16_t* ngain;  // bf16 [K]
    float* nh;              // [M][K]: h, written by the first workgroup; or null
};

constexpr int kFuseRows = kGemmWaves;  // batch rows whose norm a product forms itself (one per wavefront)
constexpr int kFuseK = 2048;           // the widest such row (the model width)
constexpr int kNormPad = 8;            // bf16 padding per LDS row (spreads the rows over the banks)

template <int EPI, bool NORM = false>
__global__ __launch_bounds__(kW * kGemmWaves) void pred_gemm(Gemm g) {
    __shared__ f32x4 red[kGemmWaves - 1][kRt][kW];
    extern __shared__ uint4 an4[];  // NORM: the normalized rows, [M][K + kNormPad] bf16
    const int lane = threadIdx.x & (kW - 1), w = threadIdx.x / kW;
    const int n0 = blockIdx.x * kNt, s = blockIdx.y, m0 = blockIdx.z * (kRt * 16);
    const int kq = g.ksplit / kGemmWaves;                // this wavefront's share (multiple of 32)
    const int kbeg = s * g.ksplit + w * kq;
    const int col = n0 + (lane & 15), kl = 8 * (lane >> 4);
    const uint16_t* wrow = g.w + (size_t)col * g.K + kbeg + kl;
    f32x4 acc[kRt];
#pragma unroll
    for (int r = 0; r < kRt; ++r) acc[r] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    const bool rows_in[kRt] = {m0 + (lane & 15) < g.M, m0 + 16 + (lane & 15) < g.M, m0 + 32 + (lane & 15) < g.M,
                               m0 + 48 + (lane & 15) < g.M};
    // four 32-wide steps at a time: their weight loads (the HBM stream) are
    // all issued before the first product waits, then the activation tiles
    // (read by every column tile, so cache hits) step by step
    bf16x8 bw[4];
    auto load_w = [&](int k0) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
            bw[u] = k0 + 32 * u < kq ? *reinterpret_cast<const bf16x8*>(wrow + k0 + 32 * u)
                                     : bf16x8{0, 0, 0, 0, 0, 0, 0, 0};
    };
    load_w(0);
    uint16_t* const an = reinterpret_cast<uint16_t*>(an4);
    const int pitch = g.K + kNormPad;
    if constexpr (NORM) {
        // wavefront w forms row w (while the first weights are in flight):
        // lane l holds channels 512 i + 8 l .. + 7
        if (w < g.M) {
            const int b = w;
            const bool writer = g.nh && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0;
            float hv[kFuseK / 512][8];
            float ss = 0.0f;
#pragma unroll
            for (int i = 0; i < kFuseK / 512; ++i) {
                const int c = 512 * i + 8 * lane;
#pragma unroll
                for (int j = 0; j < 8; ++j) hv[i][j] = 0.0f;
                if (c >= g.K) continue;
                if (g.nres) {
                    const float4 r0 = *reinterpret_cast<const float4*>(g.nres + (size_t)b * g.K + c);
                    const float4 r1 = *reinterpret_cast<const float4*>(g.nres + (size_t)b * g.K + c + 4);
                    hv[i][0] = r0.x; hv[i][1] = r0.y; hv[i][2] = r0.z; hv[i][3] = r0.w;
                    hv[i][4] = r1.x; hv[i][5] = r1.y; hv[i][6] = r1.z; hv[i][7] = r1.w;
                }
                // the partials four at a time, every load of a group issued
                // before its adds, which run in split order
                for (int s0 = 0; s0 < g.nsplits; s0 += 4) {
                    float4 pp[4][2];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        if (s0 + u < g.nsplits) {
                            const float* q = g.npart + ((size_t)(s0 + u) * g.M + b) * g.K + c;
                            pp[u][0] = *reinterpret_cast<const float4*>(q);
                            pp[u][1] = *reinterpret_cast<const float4*>(q + 4);
                        }
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        if (s0 + u < g.nsplits) {
                            hv[i][0] = hv[i][0] + pp[u][0].x; hv[i][1] = hv[i][1] + pp[u][0].y;
                            hv[i][2] = hv[i][2] + pp[u][0].z; hv[i][3] = hv[i][3] + pp[u][0].w;
                            hv[i][4] = hv[i][4] + pp[u][1].x; hv[i][5] = hv[i][5] + pp[u][1].y;
                            hv[i][6] = hv[i][6] + pp[u][1].z; hv[i][7] = hv[i][7] + pp[u][1].w;
                        }
                    }
                }
                if (writer) {
                    float* q = g.nh + (size_t)b * g.K + c;
                    *reinterpret_cast<float4*>(q) = make_float4(hv[i][0], hv[i][1], hv[i][2], hv[i][3]);
                    *reinterpret_cast<float4*>(q + 4) = make_float4(hv[i][4], hv[i][5], hv[i][6], hv[i][7]);
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) ss = ss + hv[i][j] * hv[i][j];
            }
            for (int o = kW / 2; o > 0; o >>= 1) ss = ss + __shfl_xor(ss, o);
            const float inv = 1.0f / __builtin_sqrtf(ss / (float)g.K + kEps);
#pragma unroll
            for (int i = 0; i < kFuseK / 512; ++i) {
                const int c = 512 * i + 8 * lane;
                if (c >= g.K) continue;
                const uint4 gw = *reinterpret_cast<const uint4*>(g.ngain + c);
                const uint32_t gv[4] = {gw.x, gw.y, gw.z, gw.w};
                uint32_t o[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint32_t lo = to_bf(hv[i][2 * j] * inv * __uint_as_float(gv[j] << 16));
                    const uint32_t hi = to_bf(hv[i][2 * j + 1] * inv * __uint_as_float(gv[j] & 0xFFFF0000u));
                    o[j] = lo | (hi << 16);
                }
                *reinterpret_cast<uint4*>(an + (size_t)b * pitch + c) = make_uint4(o[0], o[1], o[2], o[3]);
            }
        }
        __syncthreads();
    }
    for (int k0 = 0; k0 < kq; k0 += 4 * 32) {
        if (k0 > 0) load_w(k0);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (k0 + 32 * u >= kq) break;
            const int k = k0 + 32 * u;
#pragma unroll
            for (int r = 0; r < kRt; ++r) {
                bf16x8 av = bf16x8{0, 0, 0, 0, 0, 0, 0, 0};
                if constexpr (NORM) {
                    if (r == 0 && rows_in[0])
                        av = *reinterpret_cast<const bf16x8*>(an + (size_t)(lane & 15) * pitch + kbeg + kl + k);
                } else if (rows_in[r]) {
                    av = *reinterpret_cast<const bf16x8*>(g.a + (size_t)(m0 + 16 * r + (lane & 15)) * g.K + kbeg + kl + k);
                }
                acc[r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bw[u], acc[r], 0, 0, 0);
            }
        }
    }
    // the four wavefronts' sums, added in the order ((w0 + w1) + w2) + w3
    if (w > 0) {
#pragma unroll
        for (int r = 0; r < kRt; ++r) red[w - 1][r][lane] = acc[r];
    }
    __syncthreads();
    if (w != 0) return;
#pragma unroll
    for (int r = 0; r < kRt; ++r)
#pragma unroll
        for (int v = 0; v < kGemmWaves - 1; ++v) acc[r] = acc[r] + red[v][r][lane];
#pragma unroll
    for (int r = 0; r < kRt; ++r) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = m0 + 16 * r + 4 * (lane >> 4) + i;
            if (row >= g.M) continue;
            const float v = acc[r][i];
            if constexpr (EPI == kPartial) {
                g.out[((size_t)s * g.M + row) * g.N + col] = v;
            } else if constexpr (EPI == kStore) {
                g.out[(size_t)row * g.N + col] = v;
            } else if constexpr (EPI == kResidOut) {
                g.out16[(size_t)row * g.N + col] = to_bf(bf(g.resid[(size_t)row * g.N + col]) + v);
            } else {
                // interleaved rows: column 2j is gate j, 2j + 1 is up j; the
                // even lane gets its neighbour's up value
                const float up = __shfl_xor(v, 1);
                if ((col & 1) == 0) {
                    const float gate = v;
                    const float silu = gate / (1.0f + __expf(-gate));
                    g.out16[(size_t)row * (g.N / 2) + col / 2] = to_bf(silu * up);
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Residual stream update and RMSNorm of one batch row per workgroup:
// h = resid + sum_s part[s] (s in order), stored fp32, and
// n = bf16(h / sqrt(mean(h^2) + eps) * gain).
constexpr int kRowThreads = 256;

struct RowArgs {
    const float* resid;  // [M][m] or null
    const float* part;   // [splits][M][m]
    int32_t splits, M, m;
    const uint16_t* gain;  // bf16 [m]
    float* h;            // [M][m]
    uint16_t* n;         // bf16 [M][m]
};

constexpr int kMaxSplits = 16;  // hidden / 512 and ffn / 512 at their largest

__global__ __launch_bounds__(kRowThreads) void pred_row(RowArgs a) {
    __shared__ float red[kRowThreads / kW];
    const int b = blockIdx.x, t = threadIdx.x;
    float ss = 0.0f;
    for (int c = t; c < a.m; c += kRowThreads) {
        // every partial loaded before the first add, then summed in order
        float pv[kMaxSplits];
#pragma unroll
        for (int s = 0; s < kMaxSplits; ++s) pv[s] = s < a.splits ? a.part[((size_t)s * a.M + b) * a.m + c] : 0.0f;
        float v = a.resid ? a.resid[(size_t)b * a.m + c] : 0.0f;
#pragma unroll
        for (int s = 0; s < kMaxSplits; ++s)
            if (s < a.splits) v = v + pv[s];
        a.h[(size_t)b * a.m + c] = v;
        ss = ss + v * v;
    }
    // the sum of squares: a butterfly in each wavefront, then the
    // wavefronts' sums in order
    for (int o = kW / 2; o > 0; o >>= 1) ss = ss + __shfl_xor(ss, o);
    if ((t & (kW - 1)) == 0) red[t / kW] = ss;
    __syncthreads();
    float tot = red[0];
#pragma unroll
    for (int w = 1; w < kRowThreads / kW; ++w) tot = tot + red[w];
    const float inv = 1.0f / __builtin_sqrtf(tot / (float)a.m + kEps);
    for (int c = t; c < a.m; c += kRowThreads)
        a.n[(size_t)b * a.m + c] = to_bf(a.h[(size_t)b * a.m + c] * inv * bf(a.gain[c]));
}

// ---------------------------------------------------------------------------
// Attention of one (sequence, head) per wavefront.  Lane d holds channel d of
// the head: q and k get the rotary position (pairs (2i, 2i + 1) turned by
// pos * 10000^(-2i/64): the angle formed and reduced in binary64, its sine
// and cosine in binary32), k and v go to the cache slot
// pos mod W (bf16), and the output is the softmax-weighted sum of the values
// of positions max(0, pos - W + 1) .. pos, the current one taken from LDS
// (it is never read back from memory in the same launch).
//
// Scores: lane j takes position first + j (64 positions per pass), its key
// row (128 bytes) as eight 16-byte loads, against q read from LDS.  Output:
// lane d sums channels 8 (d % 8) .. 8 (d % 8) + 7 over positions d / 8,
// d / 8 + 8, ... (one 16-byte load of the value row each), then the eight
// lanes holding the same channels add their sums.
struct AttnArgs {
    const float* qkv;    // [B][3m]: q | k | v
    uint16_t* cache;     // [B][W][2][m] bf16
    const int32_t* pos;  // [B]
    int32_t B, m, heads, window;
    uint16_t* o;         // [B][m] bf16
    double theta[kHd / 2];  // 10000^(-2i/64), i < 32 (binary64, from the host's pow)
};

__device__ __forceinline__ void widen8(const uint4& v, float* f) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = __uint_as_float(w[i] << 16);
        f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
}

constexpr int kMaxWindow = 1024;

__global__ __launch_bounds__(kW) void pred_attn(AttnArgs a) {
    const int b = blockIdx.x / a.heads, hh = blockIdx.x % a.heads, d = threadIdx.x;
    const int32_t p = a.pos[b] < 0 ? 0 : a.pos[b];
    const float* row = a.qkv + (size_t)b * 3 * a.m + hh * kHd;
    float q = row[d], k = row[a.m + d];
    const float v = row[2 * a.m + d];
    {
        // the angle pos * theta_i in binary64, reduced to [-pi, pi] there (the
        // product k * 2 pi is exact to far below a binary32 ulp for any int32
        // position), then a binary32 sincos
        const double th = (double)p * a.theta[d >> 1];
        const double kTwoPi = 6.283185307179586476925;
        const float r = (float)(th - kTwoPi * rint(th / kTwoPi));
        float sn, c;
        sincosf(r, &sn, &c);
        const float qo = __shfl_xor(q, 1), ko = __shfl_xor(k, 1);
        // (a, b) -> (a cos - b sin, a sin + b cos): the even lane holds a
        q = (d & 1) ? qo * sn + q * c : q * c - qo * sn;
        k = (d & 1) ? ko * sn + k * c : k * c - ko * sn;
    }
    const uint16_t kb = to_bf(k), vb = to_bf(v);
    const int slot = p % a.window;
    const size_t rowk = (size_t)2 * a.m;  // cache elements per (sequence, slot)
    uint16_t* const base = a.cache + (size_t)b * a.window * rowk + hh * kHd;
    base[(size_t)slot * rowk + d] = kb;
    base[(size_t)slot * rowk + a.m + d] = vb;
    const int first = p - a.window + 1 < 0 ? 0 : p - a.window + 1;
    const int n = p - first + 1;
    __shared__ float qs[kHd], sc[kMaxWindow];
    __shared__ alignas(16) uint16_t kcur[kHd], vcur[kHd];
    qs[d] = q;
    kcur[d] = kb;
    vcur[d] = vb;
    __syncthreads();
    float mx = -INFINITY;
    for (int j0 = 0; j0 < n; j0 += kW) {
        const int j = j0 + d;
        if (j < n) {
            const int pp = first + j;
            const uint4* kr = pp == p ? reinterpret_cast<const uint4*>(kcur)
                                      : reinterpret_cast<const uint4*>(base + (size_t)(pp % a.window) * rowk);
            uint4 kv[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) kv[i] = kr[i];
            float acc = 0.0f;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                float kf[8];
                widen8(kv[i], kf);
#pragma unroll
                for (int e = 0; e < 8; ++e) acc = acc + qs[8 * i + e] * kf[e];
            }
            const float sdot = acc * 0.125f;  // 1 / sqrt(64)
            sc[j] = sdot;
            mx = __builtin_fmaxf(mx, sdot);
        }
    }
    for (int o = 1; o < kW; o <<= 1) mx = __builtin_fmaxf(mx, __shfl_xor(mx, o));
    __syncthreads();
    float den = 0.0f;
    for (int j = d; j < n; j += kW) {
        const float e = __expf(sc[j] - mx);
        sc[j] = e;
        den = den + e;
    }
    for (int o = 1; o < kW; o <<= 1) den = den + __shfl_xor(den, o);
    __syncthreads();
    const int t = d >> 3, cb = d & 7;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
    // positions t, t + 8, ...: eight value rows loaded before any is added
    // (the sums run in that order)
    for (int j0 = t; j0 < n; j0 += 64) {
        uint4 vv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int j = j0 + 8 * u, pp = first + j;
            vv[u] = j >= n ? uint4{0u, 0u, 0u, 0u}
                  : pp == p ? reinterpret_cast<const uint4*>(vcur)[cb]
                            : reinterpret_cast<const uint4*>(base + (size_t)(pp % a.window) * rowk + a.m)[cb];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int j = j0 + 8 * u;
            if (j >= n) break;
            float vf[8];
            widen8(vv[u], vf);
            const float w = sc[j];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] = acc[e] + w * vf[e];
        }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        acc[e] = acc[e] + __shfl_xor(acc[e], 8);
        acc[e] = acc[e] + __shfl_xor(acc[e], 16);
        acc[e] = acc[e] + __shfl_xor(acc[e], 32);
    }
    if (t == 0) {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            w[i] = (uint32_t)to_bf(acc[2 * i] / den) | ((uint32_t)to_bf(acc[2 * i + 1] / den) << 16);
        reinterpret_cast<uint4*>(a.o + (size_t)b * a.m + hh * kHd)[cb] = uint4{w[0], w[1], w[2], w[3]};
    }
}

// ---------------------------------------------------------------------------
// Host side

struct PLayout {
    uint64_t w_in, g1, w_qkv, w_o, g2, w_gu, w_down, g3, w_out, total;  // bytes
};

uint64_t up256(uint64_t v) { return (v + 255u) & ~uint64_t(255); }

bool pcfg_valid(const rac_predictor_config* c) {
    // (every K range splits into four wavefront shares of whole 32-wide steps)
    return c && c->hidden >= 512 && c->hidden <= 8192 && c->hidden % 512 == 0 && c->model >= 128 &&
           c->model <= 2048 && c->model % 128 == 0 && c->heads >= 1 && c->heads * kHd == c->model &&
           c->ffn >= 128 && c->ffn <= 8192 && c->ffn % 128 == 0 && c->window >= 1 && c->window <= 1024 &&
           c->max_batch >= 1 && c->max_batch <= 256;
}

PLayout playout(const rac_predictor_config* c) {
    const uint64_t d = c->hidden, m = c->model, f = c->ffn;
    PLayout L;
    uint64_t o = 0;
    auto take = [&](uint64_t elems) { const uint64_t at = o; o = up256(o + elems * 2u); return at; };
    L.w_in = take(m * d);
    L.g1 = take(m);
    L.w_qkv = take(3 * m * m);
    L.w_o = take(m * m);
    L.g2 = take(m);
    L.w_gu = take(2 * f * m);
    L.w_down = take(m * f);
    L.g3 = take(m);
    L.w_out = take(d * m);
    L.total = o;
    return L;
}

// K splits of the input projection: K ranges of 512 (4 wavefronts x 128)
int in_splits(const rac_predictor_config* c) { return c->hidden / 512; }
int down_splits(const rac_predictor_config* c) { return c->ffn % 512 == 0 ? c->ffn / 512 : 1; }

struct PWork {
    uint64_t part, h0, h1, h2, n, qkv, o, gg, total;
};

PWork pwork(const rac_predictor_config* c, int B) {
    const uint64_t m = c->model, f = c->ffn;
    const uint64_t S = (uint64_t)(in_splits(c) > down_splits(c) ? in_splits(c) : down_splits(c));
    PWork W;
    uint64_t o = 0;
    auto take = [&](uint64_t bytes) { const uint64_t at = o; o = up256(o + bytes); return at; };
    W.part = take(S * B * m * 4);
    W.h0 = take((uint64_t)B * m * 4);
    W.h1 = take((uint64_t)B * m * 4);
    W.h2 = take((uint64_t)B * m * 4);
    W.n = take((uint64_t)B * m * 2);
    W.qkv = take((uint64_t)B * 3 * m * 4);
    W.o = take((uint64_t)B * m * 2);
    W.gg = take((uint64_t)B * f * 2);
    W.total = o;
    return W;
}

template <int EPI>
rac_status gemm(const uint16_t* a, const uint16_t* w, int M, int N, int K, int splits, float* out, uint16_t* out16,
                const uint16_t* resid, hipStream_t st) {
    Gemm g{a, w, M, N, K, K / splits, out, out16, resid, nullptr, nullptr, 0, nullptr, nullptr};
    void* args[] = {&g};
    const dim3 grid((unsigned)(N / kNt), (unsigned)splits, (unsigned)((M + kRt * 16 - 1) / (kRt * 16)));
    return hipLaunchKernel(reinterpret_cast<const void*>(pred_gemm<EPI>), grid, dim3(kW * kGemmWaves), args, 0, st) ==
                   hipSuccess
               ? RAC_OK
               : RAC_ERR_HIP;
}

// The product of the normalized rows h = nres + sum_s npart[s] (one K range,
// M <= kFuseRows, K <= kFuseK): every workgroup forms the norm in LDS.
template <int EPI>
rac_status gemm_norm(const float* nres, const float* npart, int nsplits, const uint16_t* gain, float* nh,
                     const uint16_t* w, int M, int N, int K, float* out, uint16_t* out16, const uint16_t* resid,
                     hipStream_t st) {
    Gemm g{nullptr, w, M, N, K, K, out, out16, resid, nres, npart, nsplits, gain, nh};
    void* args[] = {&g};
    const size_t lds = (size_t)M * (size_t)(K + kNormPad) * 2u;
    return hipLaunchKernel(reinterpret_cast<const void*>(pred_gemm<EPI, true>), dim3((unsigned)(N / kNt), 1u, 1u),
                           dim3(kW * kGemmWaves), args, lds, st) == hipSuccess
               ? RAC_OK
               : RAC_ERR_HIP;
}

rac_status row(const float* resid, const float* part, int splits, int M, int m, const uint16_t* gain, float* h,
               uint16_t* n, hipStream_t st) {
    RowArgs r{resid, part, splits, M, m, gain, h, n};
    void* args[] = {&r};
    return hipLaunchKernel(reinterpret_cast<const void*>(pred_row), dim3((unsigned)M), dim3(kRowThreads), args, 0,
                           st) == hipSuccess
               ? RAC_OK
               : RAC_ERR_HIP;
}

rac_status attention(const rac_predictor_config* cfg, const float* qkv, void* cache, const int32_t* pos, int B,
                     uint16_t* o, hipStream_t st) {
    AttnArgs a{qkv, static_cast<uint16_t*>(cache), pos, B, cfg->model, cfg->heads, cfg->window, o, {}};
    for (int i = 0; i < kHd / 2; ++i) a.theta[i] = std::pow(10000.0, -2.0 * i / kHd);
    void* args[] = {&a};
    return hipLaunchKernel(reinterpret_cast<const void*>(pred_attn), dim3((unsigned)(B * cfg->heads)), dim3(kW), args,
                           0, st) == hipSuccess
               ? RAC_OK
               : RAC_ERR_HIP;
}

bool al(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

}  // namespace

extern "C" {

rac_status rac_predictor_layout(const rac_predictor_config* cfg, rac_predictor_offsets* out) {
    if (!pcfg_valid(cfg) || !out) return RAC_ERR_INVALID;
    const PLayout L = playout(cfg);
    out->w_in = L.w_in;
    out->g1 = L.g1;
    out->w_qkv = L.w_qkv;
    out->w_o = L.w_o;
    out->g2 = L.g2;
    out->w_gu = L.w_gu;
    out->w_down = L.w_down;
    out->g3 = L.g3;
    out->w_out = L.w_out;
    out->total = L.total;
    return RAC_OK;
}

size_t rac_predictor_cache_bytes(const rac_predictor_config* cfg) {
    if (!pcfg_valid(cfg)) return 0;
    return (size_t)cfg->max_batch * (size_t)cfg->window * 2u * (size_t)cfg->model * 2u;
}

size_t rac_predictor_workspace_bytes(const rac_predictor_config* cfg) {
    if (!pcfg_valid(cfg)) return 0;
    return (size_t)pwork(cfg, cfg->max_batch).total;
}

rac_status rac_predictor_step(const rac_predictor_config* cfg, const void* weights, void* cache, const int32_t* pos,
                              int32_t batch, const void* h_prev, void* ref_out, void* workspace,
                              size_t workspace_bytes, rac_stream_t stream) {
    if (!pcfg_valid(cfg) || batch < 0 || batch > cfg->max_batch) return RAC_ERR_INVALID;
    if (batch == 0) return RAC_OK;
    if (!weights || !cache || !pos || !h_prev || !ref_out || !workspace) return RAC_ERR_INVALID;
    if (!al(weights, 256) || !al(cache, 16) || !al(pos, 4) || !al(h_prev, 16) || !al(ref_out, 16) ||
        !al(workspace, 256))
        return RAC_ERR_ALIGN;
    const PWork W = pwork(cfg, cfg->max_batch);
    if (workspace_bytes < W.total) return RAC_ERR_CAPACITY;
    const PWork Wb = pwork(cfg, batch);  // (layout for this batch; fits in the max-batch one)
    const PLayout L = playout(cfg);
    const int B = batch, d = cfg->hidden, m = cfg->model, f = cfg->ffn;
    const uint8_t* wb = static_cast<const uint8_t*>(weights);
    auto wt = [&](uint64_t off) { return reinterpret_cast<const uint16_t*>(wb + off); };
    uint8_t* ws = static_cast<uint8_t*>(workspace);
    float* part = reinterpret_cast<float*>(ws + Wb.part);
    float* h0 = reinterpret_cast<float*>(ws + Wb.h0);
    float* h1 = reinterpret_cast<float*>(ws + Wb.h1);
    float* h2 = reinterpret_cast<float*>(ws + Wb.h2);
    uint16_t* n = reinterpret_cast<uint16_t*>(ws + Wb.n);
    float* qkv = reinterpret_cast<float*>(ws + Wb.qkv);
    uint16_t* o = reinterpret_cast<uint16_t*>(ws + Wb.o);
    uint16_t* gg = reinterpret_cast<uint16_t*>(ws + Wb.gg);
    const uint16_t* x = static_cast<const uint16_t*>(h_prev);
    hipStream_t st = stream;
    rac_status s;
    const int si = in_splits(cfg), sd = down_splits(cfg);
    if (B <= kFuseRows && m <= kFuseK) {
        // small batches: each norm is formed by the product that consumes
        // it (seven launches instead of ten)
        if ((s = gemm<kPartial>(x, wt(L.w_in), B, m, d, si, part, nullptr, nullptr, st)) != RAC_OK) return s;
        if ((s = gemm_norm<kStore>(nullptr, part, si, wt(L.g1), h0, wt(L.w_qkv), B, 3 * m, m, qkv, nullptr, nullptr,
                                   st)) != RAC_OK)
            return s;
        if ((s = attention(cfg, qkv, cache, pos, B, o, st)) != RAC_OK) return s;
        if ((s = gemm<kPartial>(o, wt(L.w_o), B, m, m, 1, part, nullptr, nullptr, st)) != RAC_OK) return s;
        if ((s = gemm_norm<kSwiglu>(h0, part, 1, wt(L.g2), h1, wt(L.w_gu), B, 2 * f, m, nullptr, gg, nullptr, st)) !=
            RAC_OK)
            return s;
        if ((s = gemm<kPartial>(gg, wt(L.w_down), B, m, f, sd, part, nullptr, nullptr, st)) != RAC_OK) return s;
        return gemm_norm<kResidOut>(h1, part, sd, wt(L.g3), nullptr, wt(L.w_out), B, d, m, nullptr,
                                    static_cast<uint16_t*>(ref_out), x, st);
    }
    // h0 = x W_in^T (split K), then n1 = RMSNorm(h0)
    if ((s = gemm<kPartial>(x, wt(L.w_in), B, m, d, si, part, nullptr, nullptr, st)) != RAC_OK) return s;
    if ((s = row(nullptr, part, si, B, m, wt(L.g1), h0, n, st)) != RAC_OK) return s;
    // q, k, v; attention over the window; h1 = h0 + o W_o^T; n2 = RMSNorm(h1)
    if ((s = gemm<kStore>(n, wt(L.w_qkv), B, 3 * m, m, 1, qkv, nullptr, nullptr, st)) != RAC_OK) return s;
    if ((s = attention(cfg, qkv, cache, pos, B, o, st)) != RAC_OK) return s;
    if ((s = gemm<kPartial>(o, wt(L.w_o), B, m, m, 1, part, nullptr, nullptr, st)) != RAC_OK) return s;
    if ((s = row(h0, part, 1, B, m, wt(L.g2), h1, n, st)) != RAC_OK) return s;
    // SwiGLU; h2 = h1 + g W_down^T; n3 = RMSNorm(h2)
    if ((s = gemm<kSwiglu>(n, wt(L.w_gu), B, 2 * f, m, 1, nullptr, gg, nullptr, st)) != RAC_OK) return s;
    if ((s = gemm<kPartial>(gg, wt(L.w_down), B, m, f, sd, part, nullptr, nullptr, st)) != RAC_OK) return s;
    if ((s = row(h1, part, sd, B, m, wt(L.g3), h2, n, st)) != RAC_OK) return s;
    // R = x + n3 W_out^T (bf16)
    return gemm<kResidOut>(n, wt(L.w_out), B, d, m, 1, nullptr, static_cast<uint16_t*>(ref_out), x, st);
}

}  // extern "C"
