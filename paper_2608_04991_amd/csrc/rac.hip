// rac.hip - gfx950 kernels and C ABI of the RAC aligned residual codec.
//
// Method: the paper's Section "Quality- and Cost-Constrained Aligned Residual
// Encoding" (Eq. affine-fit, Eq. aligned-residual, Eq. residual-quantization,
// the outlier paragraph, Eq. residual-reconstruction).  The contract of every
// entry point is documented in include/rac.h.
//
// Mapping onto CDNA4.  The codec is a per-token-row stream with no dense
// contraction, so it is HBM-bound and uses no MFMA.  One 64-lane wavefront
// owns one token row.  A row is cut into 512-channel chunks; in chunk `it`,
// lane l holds channels [it*512 + 8l, it*512 + 8l + 8) -- one 128-bit load of
// x and one of ref per lane and chunk, fully coalesced (1 KiB per wave load).
// The whole row stays in VGPRs: fit, residual, outlier choice, scale,
// quantization, packing and the fused sender reconstruction all run on
// registers, and every byte of x/ref is read from HBM exactly once and every
// output byte written exactly once.
//
// Exactness.  The sums of the fit follow a fixed pairwise tree over channel
// order: a lane-local tree over its 8 contiguous channels, then a butterfly
// across lanes whose every step adds the partial sums of two adjacent
// aligned blocks (DPP quad_perm / row_half_mirror / row_mirror, then
// v_permlane16_swap and v_permlane32_swap), then a tree over chunks.  Since
// floating-point addition is commutative, that reproduces the canonical
// pairwise sum exactly.  The file is compiled with -ffp-contract=off so no
// multiply-add is fused, and divisions stay correctly rounded.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rac.h"

namespace {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kBlock = kWave * kWavesPerBlock;
constexpr int kChunk = 512;
constexpr float kMagic = 12582912.0f;  // 1.5 * 2^23: adding it rounds to an integer (RNE)
// Quotients t' = E * (1/s) within this distance of a half-integer are
// recomputed with the correctly rounded division E / s.  |t' - E/s| is below
// 2 ulp(128) = 2^-16 for |t'| <= 128, so the fast rounding is exact elsewhere.
constexpr float kNearHalf = 0.5f - 0x1p-14f;

struct alignas(8) Args {
    const uint16_t* x;
    const uint16_t* ref;
    const float* steps;
    uint8_t* wire;
    void* xhat;
    uint64_t off_coef, off_scale, off_codes, off_outl, total;
    uint64_t end_coef, end_scale, end_codes, end_outl;  // first byte after each section
    int64_t tokens;
    int32_t d;
    int32_t nch;        // chunks per row: ceil(d / 512)
    int32_t ga, gq;     // group sizes
    int32_t lane_lv_a;  // butterfly levels inside a chunk: log2(min(g, 512) / 8)
    int32_t lane_lv_q;
    int32_t cpg_a;      // chunks per group: max(1, g / 512)
    int32_t cpg_q;
    int32_t k;
    int32_t fixed;
    int32_t xhat_bf16;
    int32_t write_header;
    uint32_t hdr[24];   // first 96 bytes of the header; the rest is zero
};

// ---------------------------------------------------------------------------
// Number formats

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ void widen8(const uint4& w, float* v) {
    v[0] = bf16_lo(w.x); v[1] = bf16_hi(w.x); v[2] = bf16_lo(w.y); v[3] = bf16_hi(w.y);
    v[4] = bf16_lo(w.z); v[5] = bf16_hi(w.z); v[6] = bf16_lo(w.w); v[7] = bf16_hi(w.w);
}

// fp32 -> fp16 pattern, round to nearest even, magnitudes above 65504 clamp.
__device__ __forceinline__ uint32_t f16_rne_sat(float v) {
    v = __builtin_fminf(__builtin_fmaxf(v, -65504.0f), 65504.0f);
    const _Float16 h = (_Float16)v;
    return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

__device__ __forceinline__ float f16_value(uint32_t bits) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits);
}

// fp32 -> bf16 pattern, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t bf16_rne(float v) {
    const uint32_t u = __float_as_uint(v);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Smallest positive fp16 h with value(h) * q >= m  (m > 0); 0x7BFF if none.
// value(h) * q is exact in binary32, so the test is an exact comparison.  The
// start point RNE(m / q) is within one fp16 step of the answer.
__device__ __forceinline__ uint32_t scale_roundup(float m, float q) {
    if (m > 65504.0f * q) return 0x7BFFu;
    uint32_t h = f16_rne_sat(m / q);
    if (h == 0u) h = 1u;
#pragma unroll
    for (int i = 0; i < 3; ++i)
        if (h < 0x7BFFu && f16_value(h) * q < m) ++h;
#pragma unroll
    for (int i = 0; i < 3; ++i)
        if (h > 1u && f16_value(h - 1u) * q >= m) --h;
    return h;
}

// Smallest positive fp16 h with value(h) >= step; 0x7BFF above 65504.
__device__ __forceinline__ uint32_t step_roundup(float step) {
    if (!(step <= 65504.0f)) return 0x7BFFu;
    uint32_t h = f16_rne_sat(step);
    if (h == 0u || (h & 0x8000u)) h = 1u;
#pragma unroll
    for (int i = 0; i < 3; ++i)
        if (h < 0x7BFFu && f16_value(h) < step) ++h;
#pragma unroll
    for (int i = 0; i < 3; ++i)
        if (h > 1u && f16_value(h - 1u) >= step) --h;
    return h;
}

// Closed-form least squares of one group from its centred moments:
// alpha* = C_rx / C_rr, beta* = m_x - alpha* m_r; a zero-variance reference
// gives (0, m_x).  Returns the fp16 pair (alpha | beta << 16).
__device__ __forceinline__ uint32_t fit_coef(float crr, float crx, float mr, float mx) {
    float as, bs;
    if (crr == 0.0f) {
        as = 0.0f;
        bs = mx;
    } else {
        as = crx / crr;
        bs = mx - as * mr;
    }
    return f16_rne_sat(as) | (f16_rne_sat(bs) << 16);
}

// E = x - R~ with R~ = alpha r + beta from the serialized pair (two roundings).
__device__ __forceinline__ void residual8(uint32_t cf, const float* r, const float* x, float* e) {
    const float a = f16_value(cf & 0xFFFFu), b0 = f16_value(cf >> 16);
#pragma unroll
    for (int j = 0; j < 8; ++j) e[j] = x[j] - (a * r[j] + b0);
}

// ---------------------------------------------------------------------------
// Cross-lane partner of the adjacent aligned block at butterfly level `lv`
// (level lv merges blocks of 2^lv lanes into blocks of 2^(lv+1)).

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// Sum of the two halves of a 32-lane (lv 4) or 64-lane (lv 5) block.
__device__ __forceinline__ float pair16_sum(float v) {
    auto p = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(int, v),
                                              __builtin_bit_cast(int, v), false, false);
    return __builtin_bit_cast(float, (int)p[0]) + __builtin_bit_cast(float, (int)p[1]);
}
__device__ __forceinline__ float pair32_sum(float v) {
    auto p = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(int, v),
                                              __builtin_bit_cast(int, v), false, false);
    return __builtin_bit_cast(float, (int)p[0]) + __builtin_bit_cast(float, (int)p[1]);
}
__device__ __forceinline__ float pair16_max(float v) {
    auto p = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(int, v),
                                              __builtin_bit_cast(int, v), false, false);
    return __builtin_fmaxf(__builtin_bit_cast(float, (int)p[0]),
                           __builtin_bit_cast(float, (int)p[1]));
}
__device__ __forceinline__ float pair32_max(float v) {
    auto p = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(int, v),
                                              __builtin_bit_cast(int, v), false, false);
    return __builtin_fmaxf(__builtin_bit_cast(float, (int)p[0]),
                           __builtin_bit_cast(float, (int)p[1]));
}

// Pairwise sum across the 2^levels lanes of an aligned lane block.
__device__ __forceinline__ float lane_sum(float v, int levels) {
    if (levels > 0) v = v + dpp<0xB1>(v);    // quad_perm [1,0,3,2]
    if (levels > 1) v = v + dpp<0x4E>(v);    // quad_perm [2,3,0,1]
    if (levels > 2) v = v + dpp<0x141>(v);   // row_half_mirror
    if (levels > 3) v = v + dpp<0x140>(v);   // row_mirror
    if (levels > 4) v = pair16_sum(v);
    if (levels > 5) v = pair32_sum(v);
    return v;
}

__device__ __forceinline__ float lane_max(float v, int levels) {
    if (levels > 0) v = __builtin_fmaxf(v, dpp<0xB1>(v));
    if (levels > 1) v = __builtin_fmaxf(v, dpp<0x4E>(v));
    if (levels > 2) v = __builtin_fmaxf(v, dpp<0x141>(v));
    if (levels > 3) v = __builtin_fmaxf(v, dpp<0x140>(v));
    if (levels > 4) v = pair16_max(v);
    if (levels > 5) v = pair32_max(v);
    return v;
}

__device__ __forceinline__ float tree8(const float* v) {
    return ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
}

// Pairwise tree over the chunks of groups spanning `cpg` chunks, then the
// group total broadcast back to each of its chunks.
template <int MAXCH>
__device__ __forceinline__ void chunk_tree_sum(float* s, int cpg) {
    constexpr int kLevels = MAXCH >= 16 ? 4 : MAXCH >= 8 ? 3 : MAXCH >= 4 ? 2 : MAXCH >= 2 ? 1 : 0;
#pragma unroll
    for (int lv = 0; lv < kLevels; ++lv) {
        const int w = 1 << lv;
        if (w < cpg) {
#pragma unroll
            for (int it = 0; it + w < MAXCH; it += 2 * w) s[it] = s[it] + s[it + w];
        }
    }
#pragma unroll
    for (int lv = kLevels - 1; lv >= 0; --lv) {
        const int w = 1 << lv;
        if (w < cpg) {
#pragma unroll
            for (int it = 0; it + w < MAXCH; it += 2 * w) s[it + w] = s[it];
        }
    }
}

template <int MAXCH>
__device__ __forceinline__ void chunk_tree_max(float* s, int cpg) {
    constexpr int kLevels = MAXCH >= 16 ? 4 : MAXCH >= 8 ? 3 : MAXCH >= 4 ? 2 : MAXCH >= 2 ? 1 : 0;
#pragma unroll
    for (int lv = 0; lv < kLevels; ++lv) {
        const int w = 1 << lv;
        if (w < cpg) {
#pragma unroll
            for (int it = 0; it + w < MAXCH; it += 2 * w) s[it] = __builtin_fmaxf(s[it], s[it + w]);
        }
    }
#pragma unroll
    for (int lv = kLevels - 1; lv >= 0; --lv) {
        const int w = 1 << lv;
        if (w < cpg) {
#pragma unroll
            for (int it = 0; it + w < MAXCH; it += 2 * w) s[it + w] = s[it];
        }
    }
}

__device__ __forceinline__ uint32_t mbcnt64(uint64_t m) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }

__device__ __forceinline__ uint32_t rdlane(uint32_t v, int l) {
    return (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

// Wave-wide max of unsigned values (all lanes get it).
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    float f = __uint_as_float(v);  // order-preserving for non-NaN patterns < 0x7F800000
    f = lane_max(f, 6);
    return __float_as_uint(f);
}

// One bit per (chunk, channel-in-lane) slot of a lane: bit it*8 + j.
template <int MAXCH>
struct SlotMask {
    static constexpr int kWords = (MAXCH * 8 + 63) / 64;
    uint64_t w[kWords];
    __device__ __forceinline__ bool test(int slot) const {  // slot is a compile-time constant
        return (w[slot / 64] >> (slot % 64)) & 1ull;
    }
    __device__ __forceinline__ void set(int slot) {        // slot may be a runtime value
#pragma unroll
        for (int i = 0; i < kWords; ++i)
            if ((slot >> 6) == i) w[i] |= 1ull << (slot & 63);
    }
};

// ---------------------------------------------------------------------------
// Header and inter-section padding (written by wave 0 of block 0).

__device__ __forceinline__ void zero_bytes(uint8_t* w, uint64_t lo, uint64_t hi, uint32_t lane) {
    for (uint64_t p = lo + lane; p < hi; p += kWave) w[p] = 0;
}

__device__ __forceinline__ void write_header(const Args& A, uint32_t lane) {
    uint32_t* w32 = reinterpret_cast<uint32_t*>(A.wire);
    // header fields (static indices: a dynamic index would spill the whole
    // argument block to scratch), then zeros up to 256 bytes
    if (lane == 0) {
#pragma unroll
        for (int i = 0; i < 24; ++i) w32[i] = A.hdr[i];
    }
    if (lane >= 24) w32[lane] = 0u;
    zero_bytes(A.wire, A.end_coef, A.off_scale, lane);
    zero_bytes(A.wire, A.end_scale, A.off_codes, lane);
    zero_bytes(A.wire, A.end_codes, A.off_outl, lane);
    zero_bytes(A.wire, A.end_outl, A.total, lane);
}

// ---------------------------------------------------------------------------
// Code packing of one lane's 8 channels of one chunk.

template <int BITS>
struct Packed;
template <>
struct Packed<2> { uint32_t w; };   // 16 bits used
template <>
struct Packed<3> { uint32_t w; };   // 24 bits used
template <>
struct Packed<4> { uint32_t w; };
template <>
struct Packed<8> { uint32_t lo, hi; };

template <int BITS>
__device__ __forceinline__ void pack_put(Packed<BITS>& p, int j, uint32_t code_bits);

template <>
__device__ __forceinline__ void pack_put<2>(Packed<2>& p, int j, uint32_t c) { p.w |= (c & 3u) << (2 * j); }
template <>
__device__ __forceinline__ void pack_put<3>(Packed<3>& p, int j, uint32_t c) { p.w |= (c & 7u) << (3 * j); }
template <>
__device__ __forceinline__ void pack_put<4>(Packed<4>& p, int j, uint32_t c) { p.w |= (c & 15u) << (4 * j); }
template <>
__device__ __forceinline__ void pack_put<8>(Packed<8>& p, int j, uint32_t c) {
    if (j < 4) p.lo |= (c & 255u) << (8 * j);
    else p.hi |= (c & 255u) << (8 * (j - 4));
}

// Store the packed codes of chunk `it` for this lane.  Lane l's 8 channels
// occupy bytes [l*BITS, l*BITS + BITS) of the chunk's 64*BITS bytes.
template <int BITS>
__device__ __forceinline__ void store_codes(uint8_t* row_codes, int it, uint32_t lane, bool active,
                                            bool dword_ok, const Packed<BITS>& p);

template <>
__device__ __forceinline__ void store_codes<2>(uint8_t* rc, int it, uint32_t lane, bool active, bool,
                                               const Packed<2>& p) {
    if (active) *reinterpret_cast<uint16_t*>(rc + it * 128 + lane * 2) = (uint16_t)p.w;
}
template <>
__device__ __forceinline__ void store_codes<4>(uint8_t* rc, int it, uint32_t lane, bool active, bool,
                                               const Packed<4>& p) {
    if (active) *reinterpret_cast<uint32_t*>(rc + it * 256 + lane * 4) = p.w;
}
template <>
__device__ __forceinline__ void store_codes<8>(uint8_t* rc, int it, uint32_t lane, bool active, bool,
                                               const Packed<8>& p) {
    if (active) *reinterpret_cast<uint2*>(rc + it * 512 + lane * 8) = make_uint2(p.lo, p.hi);
}
template <>
__device__ __forceinline__ void store_codes<3>(uint8_t* rc, int it, uint32_t lane, bool active,
                                               bool dword_ok, const Packed<3>& p) {
    // Four lanes own 96 contiguous bits = 3 dwords; lane j of the quad writes
    // dword j from its own 24 bits and the next lane's.
    const uint32_t nxt = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)p.w, 0x39 /* quad_perm [1,2,3,0] */,
                                                               0xF, 0xF, false);
    uint8_t* base = rc + it * 192;
    if (dword_ok) {
        const uint32_t j = lane & 3u;
        const uint32_t dw = j == 0 ? (p.w | (nxt << 24))
                          : j == 1 ? ((p.w >> 8) | (nxt << 16))
                                   : ((p.w >> 16) | (nxt << 8));
        if (active && j < 3u) *reinterpret_cast<uint32_t*>(base + ((lane >> 2) * 3u + j) * 4u) = dw;
    } else if (active) {
        base[lane * 3 + 0] = (uint8_t)p.w;
        base[lane * 3 + 1] = (uint8_t)(p.w >> 8);
        base[lane * 3 + 2] = (uint8_t)(p.w >> 16);
    }
}

// Load this lane's packed codes of chunk `it` (inverse of store_codes).
template <int BITS>
__device__ __forceinline__ void load_codes(const uint8_t* rc, int it, uint32_t lane, bool active,
                                           bool dword_ok, uint32_t& lo, uint32_t& hi) {
    lo = hi = 0;
    if (!active) return;
    if constexpr (BITS == 2) {
        lo = *reinterpret_cast<const uint16_t*>(rc + it * 128 + lane * 2);
    } else if constexpr (BITS == 4) {
        lo = *reinterpret_cast<const uint32_t*>(rc + it * 256 + lane * 4);
    } else if constexpr (BITS == 8) {
        const uint2 v = *reinterpret_cast<const uint2*>(rc + it * 512 + lane * 8);
        lo = v.x;
        hi = v.y;
    } else {
        const uint8_t* base = rc + it * 192;
        if (dword_ok) {
            const uint32_t j = lane & 3u;
            const uint32_t* dws = reinterpret_cast<const uint32_t*>(base) + (lane >> 2) * 3u;
            // lane j's 24 bits start at bit 24j of the quad's 96 bits
            const uint32_t w0 = dws[(24u * j) >> 5];
            const uint32_t w1 = j == 3u ? 0u : dws[((24u * j) >> 5) + 1u];
            const uint32_t sh = (24u * j) & 31u;
            lo = (sh ? ((w0 >> sh) | (w1 << (32u - sh))) : w0) & 0xFFFFFFu;
        } else {
            lo = (uint32_t)base[lane * 3] | ((uint32_t)base[lane * 3 + 1] << 8) |
                 ((uint32_t)base[lane * 3 + 2] << 16);
        }
    }
}

template <int BITS>
__device__ __forceinline__ int32_t code_at(uint32_t lo, uint32_t hi, int j) {
    uint32_t u;
    if constexpr (BITS == 8) u = j < 4 ? (lo >> (8 * j)) : (hi >> (8 * (j - 4)));
    else u = lo >> (BITS * j);
    return ((int32_t)(u << (32 - BITS))) >> (32 - BITS);  // sign-extend
}

// max |E| over the lane's 8 channels of chunk `it`, outliers counted as 0.
template <int MAXCH>
__device__ __forceinline__ float dense_absmax8(const float* e, const SlotMask<MAXCH>& selbits,
                                               const SlotMask<MAXCH>& slot_any, int it) {
    float m = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        float v = e[j];
        if (slot_any.test(it * 8 + j))
            if (selbits.test(it * 8 + j)) v = 0.0f;
        m = __builtin_fmaxf(m, __builtin_fabsf(v));
    }
    return m;
}

__device__ __forceinline__ void store_xhat(const Args& A, uint64_t off, const float* H) {
    if (A.xhat_bf16) {
        uint4 o;
        o.x = bf16_rne(H[0]) | (bf16_rne(H[1]) << 16);
        o.y = bf16_rne(H[2]) | (bf16_rne(H[3]) << 16);
        o.z = bf16_rne(H[4]) | (bf16_rne(H[5]) << 16);
        o.w = bf16_rne(H[6]) | (bf16_rne(H[7]) << 16);
        *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(A.xhat) + off) = o;
    } else {
        float* o = reinterpret_cast<float*>(A.xhat) + off;
        *reinterpret_cast<float4*>(o) = make_float4(H[0], H[1], H[2], H[3]);
        *reinterpret_cast<float4*>(o + 4) = make_float4(H[4], H[5], H[6], H[7]);
    }
}

// ---------------------------------------------------------------------------
// Outlier choice for one row: the k largest |E| (ties to the lower channel).
//
// 1. L = k-th largest of the 64 per-lane maxima of |E|.  At least k elements
//    satisfy |E| >= L, so the k-th largest element is >= L.
// 2. Elements with |E| >= L are gathered into LDS (typically ~k of them).
// 3a. If at most 64 were gathered, the key (|E|, -channel) of each candidate
//     is ranked against the others; the candidate ranked k-1 gives the
//     threshold key (T, c*).
// 3b. Otherwise (heavy ties), T is found by bisection on the bit pattern of
//     |E| and c* by bisection on the channel among the elements equal to T.
// 4. An element is an outlier iff |E| > T, or |E| == T and channel <= c*.
//    It is marked in `selbits` (bit it*8+j of the owning lane) and in the
//    wave-uniform `slot_any`; the k outliers are gathered and written in
//    ascending channel order.

template <int MAXCH>
__device__ __forceinline__ void select_outliers(const Args& A, const float (&E)[MAXCH][8], int64_t row, uint32_t lane,
                                uint32_t* s_val, uint32_t* s_idx, SlotMask<MAXCH>& selbits,
                                SlotMask<MAXCH>& slot_any) {
    const int k = A.k, d = A.d, nch = A.nch;
    // 1. per-lane max and its rank among lanes
    float lm = 0.0f;
#pragma unroll
    for (int it = 0; it < MAXCH; ++it)
        if (it < nch && it * kChunk + (int)lane * 8 < d) {
#pragma unroll
            for (int j = 0; j < 8; ++j) lm = __builtin_fmaxf(lm, __builtin_fabsf(E[it][j]));
        }
    const uint32_t lmb = __float_as_uint(lm);
    uint32_t ge = 0;
#pragma unroll 1
    for (int l = 0; l < kWave; ++l) ge += (rdlane(lmb, l) >= lmb) ? 1u : 0u;
    const uint32_t L = wave_max_u32(ge >= (uint32_t)k ? lmb : 0u);
    const float Lf = __uint_as_float(L);

    // 2. gather candidates |E| >= L
    uint32_t ncand = 0;
#pragma unroll
    for (int it = 0; it < MAXCH; ++it)
        if (it < nch) {
            const bool act = it * kChunk + (int)lane * 8 < d;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const bool p = act && __builtin_fabsf(E[it][j]) >= Lf;
                const uint64_t m = ballot(p);
                if (m) {
                    const uint32_t pos = ncand + mbcnt64(m);
                    if (p && pos < (uint32_t)kWave) {
                        s_val[pos] = __float_as_uint(E[it][j]);
                        s_idx[pos] = (uint32_t)(it * kChunk + lane * 8 + j);
                    }
                    ncand += (uint32_t)__builtin_popcountll(m);
                }
            }
        }
    wave_lds_sync();

    uint32_t T;          // threshold |E| bits
    uint32_t cstar;      // last tied channel taken (only used when ties)
    bool ties;
    if (ncand <= (uint32_t)kWave) {
        // 3a. rank the candidate keys
        const bool have = lane < ncand;
        const uint32_t vb = have ? (s_val[lane] & 0x7FFFFFFFu) : 0u;
        const uint32_t ix = have ? s_idx[lane] : 0xFFFFu;
        const uint64_t key = have ? (((uint64_t)vb << 16) | (uint64_t)(0xFFFFu - ix)) : 0ull;
        uint32_t rank = 0;
        for (uint32_t l = 0; l < ncand; ++l) {
            const uint64_t o = ((uint64_t)rdlane((uint32_t)(key >> 32), (int)l) << 32) |
                               (uint64_t)rdlane((uint32_t)key, (int)l);
            rank += (o > key) ? 1u : 0u;
        }
        const uint64_t at = ballot(have && rank == (uint32_t)(k - 1));
        const int src = at ? (int)__builtin_ctzll(at) : 0;
        T = rdlane(vb, src);
        cstar = rdlane(ix, src);
        ties = __builtin_popcountll(ballot(have && vb >= T)) != (unsigned)k;
    } else {
        // 3b. bisection: largest T with count(|E| >= T) >= k
        // (compares are written two-sided on E so that nothing per element is
        // loop-invariant and hoisted into extra registers)
        uint32_t lo = 0u, hi = 0x7F800000u;
        while (lo < hi) {
            const uint32_t mid = lo + ((hi - lo + 1u) >> 1);
            const float mf = __uint_as_float(mid);
            uint32_t cnt = 0;
#pragma unroll
            for (int it = 0; it < MAXCH; ++it)
                if (it < nch) {
                    const bool act = it * kChunk + (int)lane * 8 < d;
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        cnt += (uint32_t)__builtin_popcountll(
                            ballot(act && (E[it][j] >= mf || E[it][j] <= -mf)));
                }
            if (cnt >= (uint32_t)k) lo = mid;
            else hi = mid - 1u;
        }
        T = lo;
        const float Tf = __uint_as_float(T);
        uint32_t gt = 0, ge2 = 0;
#pragma unroll
        for (int it = 0; it < MAXCH; ++it)
            if (it < nch) {
                const bool act = it * kChunk + (int)lane * 8 < d;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    gt += (uint32_t)__builtin_popcountll(ballot(act && (E[it][j] > Tf || E[it][j] < -Tf)));
                    ge2 += (uint32_t)__builtin_popcountll(ballot(act && (E[it][j] >= Tf || E[it][j] <= -Tf)));
                }
            }
        ties = ge2 != (uint32_t)k;
        // smallest channel c* with count(|E| == T, channel <= c*) == k - gt
        const uint32_t need = (uint32_t)k - gt;
        uint32_t clo = 0u, chi = (uint32_t)d - 1u;
        const uint32_t lane8 = lane * 8u;
        while (clo < chi) {
            const uint32_t mid = (clo + chi) >> 1;
            uint32_t cnt = 0;
#pragma unroll
            for (int it = 0; it < MAXCH; ++it)
                if (it < nch) {
                    const bool act = it * kChunk + (int)lane * 8 < d;
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        // channel it*512 + 8*lane + j <= mid, as a compare of lane8
                        const int lim = (int)mid - it * kChunk - j;
                        cnt += (uint32_t)__builtin_popcountll(ballot(
                            act && (E[it][j] == Tf || E[it][j] == -Tf) && (int)lane8 <= lim));
                    }
                }
            if (cnt >= need) chi = mid;
            else clo = mid + 1u;
        }
        cstar = clo;
    }
    wave_lds_sync();

    // 4. mark and gather the k outliers
    const float Tf = __uint_as_float(T);
    uint32_t n = 0;
#pragma unroll
    for (int it = 0; it < MAXCH; ++it)
        if (it < nch) {
            const bool act = it * kChunk + (int)lane * 8 < d;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float a = __builtin_fabsf(E[it][j]);
                const uint32_t c = (uint32_t)(it * kChunk) + lane * 8u + (uint32_t)j;
                const bool p = act && (ties ? (a > Tf || (a == Tf && c <= cstar)) : (a >= Tf));
                const uint64_t m = ballot(p);
                if (m) {
                    slot_any.set(it * 8 + j);
                    if (p) {
                        selbits.set(it * 8 + j);
                        const uint32_t pos = n + mbcnt64(m);
                        if (pos < (uint32_t)kWave) {
                            s_val[pos] = __float_as_uint(E[it][j]);
                            s_idx[pos] = c;
                        }
                    }
                    n += (uint32_t)__builtin_popcountll(m);
                }
            }
        }
    wave_lds_sync();
    // n == k here.  Lane i < k holds gathered outlier i; its output slot is
    // the number of gathered outliers with a lower channel.
    if (lane < (uint32_t)k) {
        const uint32_t c = s_idx[lane];
        const uint32_t v = s_val[lane];
        uint32_t slot = 0;
        for (int i = 0; i < k; ++i) slot += (s_idx[i] < c) ? 1u : 0u;
        uint32_t* out = reinterpret_cast<uint32_t*>(A.wire + A.off_outl) + (uint64_t)row * (uint64_t)k;
        out[slot] = c | (f16_rne_sat(__uint_as_float(v)) << 16);
    }
    wave_lds_sync();
}

// ---------------------------------------------------------------------------
// Encode with fused sender reconstruction: one wavefront per token row.

template <int BITS, int MAXCH>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(2))) void rac_encode_kernel(Args A) {
    __shared__ uint32_t s_val_all[kWavesPerBlock][kWave];
    __shared__ uint32_t s_idx_all[kWavesPerBlock][kWave];
    const uint32_t lane = threadIdx.x & (kWave - 1);
    const uint32_t wv = threadIdx.x / kWave;
    if (A.write_header && blockIdx.x == 0 && wv == 0) write_header(A, lane);
    const int64_t row = (int64_t)blockIdx.x * kWavesPerBlock + wv;
    if (row >= A.tokens) return;

    const int d = A.d, nch = A.nch;
    const float q = (float)((1 << (BITS - 1)) - 1);
    const uint64_t rbase = (uint64_t)row * (uint64_t)d;

    // a1: load x and ref rows (raw bf16 words; widening to fp32 is exact and
    // is redone where a value is needed, which keeps the row in 64 VGPRs)
    uint4 XV[MAXCH], RV[MAXCH];
#pragma unroll
    for (int it = 0; it < MAXCH; ++it) {
        XV[it] = make_uint4(0, 0, 0, 0);
        RV[it] = make_uint4(0, 0, 0, 0);
        const int c0 = it * kChunk + (int)lane * 8;
        if (it < nch && c0 < d) {
            XV[it] = *reinterpret_cast<const uint4*>(A.x + rbase + c0);
            if (A.ref) RV[it] = *reinterpret_cast<const uint4*>(A.ref + rbase + c0);
        }
    }

    // a2-a3: grouped affine fit (two-pass centred moments, pairwise sums),
    // serialized to fp16, then the residual E = x - (alpha r + beta).
    uint32_t* coef_row = reinterpret_cast<uint32_t*>(A.wire + A.off_coef) + (uint64_t)row * (uint64_t)(d / A.ga);
    const float inv_ga = 1.0f / (float)A.ga;  // exact: power of two
    float X[MAXCH][8];   // becomes the residual E
    uint32_t CF[MAXCH];  // serialized (alpha, beta) of the lane's group
    if (A.cpg_a == 1) {
        // groups lie inside one chunk: fit and residual chunk by chunk
        const int lanes_pg = A.ga >= kChunk ? kWave : A.ga / 8;
#pragma unroll
        for (int it = 0; it < MAXCH; ++it) {
            float r[8], x[8];
            widen8(RV[it], r);
            widen8(XV[it], x);
            const float mr = lane_sum(tree8(r), A.lane_lv_a) * inv_ga;
            const float mx = lane_sum(tree8(x), A.lane_lv_a) * inv_ga;
            float uu[8], uv[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float u = r[j] - mr;
                const float v = x[j] - mx;
                uu[j] = u * u;
                uv[j] = u * v;
            }
            const float crr = lane_sum(tree8(uu), A.lane_lv_a);
            const float crx = lane_sum(tree8(uv), A.lane_lv_a);
            CF[it] = fit_coef(crr, crx, mr, mx);
            const int c0 = it * kChunk + (int)lane * 8;
            if (it < nch && c0 < d && (int)lane % lanes_pg == 0) coef_row[c0 / A.ga] = CF[it];
            residual8(CF[it], r, x, X[it]);
        }
    } else {
        // groups span cpg_a chunks: chunk partial sums combined by a tree
        float SR[MAXCH], SX[MAXCH], SUU[MAXCH], SUV[MAXCH];
#pragma unroll
        for (int it = 0; it < MAXCH; ++it) {
            float r[8], x[8];
            widen8(RV[it], r);
            widen8(XV[it], x);
            SR[it] = lane_sum(tree8(r), 6);
            SX[it] = lane_sum(tree8(x), 6);
        }
        chunk_tree_sum<MAXCH>(SR, A.cpg_a);
        chunk_tree_sum<MAXCH>(SX, A.cpg_a);
#pragma unroll
        for (int it = 0; it < MAXCH; ++it) {
            const float mr = SR[it] * inv_ga, mx = SX[it] * inv_ga;
            float r[8], x[8], uu[8], uv[8];
            widen8(RV[it], r);
            widen8(XV[it], x);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float u = r[j] - mr;
                const float v = x[j] - mx;
                uu[j] = u * u;
                uv[j] = u * v;
            }
            SUU[it] = lane_sum(tree8(uu), 6);
            SUV[it] = lane_sum(tree8(uv), 6);
        }
        chunk_tree_sum<MAXCH>(SUU, A.cpg_a);
        chunk_tree_sum<MAXCH>(SUV, A.cpg_a);
#pragma unroll
        for (int it = 0; it < MAXCH; ++it) {
            CF[it] = fit_coef(SUU[it], SUV[it], SR[it] * inv_ga, SX[it] * inv_ga);
            if (it < nch && lane == 0 && (it % A.cpg_a) == 0) coef_row[(it * kChunk) / A.ga] = CF[it];
            float r[8], x[8];
            widen8(RV[it], r);
            widen8(XV[it], x);
            residual8(CF[it], r, x, X[it]);
        }
    }

    // a4: outliers
    SlotMask<MAXCH> selbits{}, slot_any{};
    if (A.k > 0) select_outliers<MAXCH>(A, X, row, lane, s_val_all[wv], s_idx_all[wv], selbits, slot_any);

    // a5: dense max per quantization group (groups spanning chunks need all
    // chunk maxima first; groups inside a chunk are done chunk by chunk)
    float M[MAXCH];
    if (A.cpg_q > 1) {
#pragma unroll
        for (int it = 0; it < MAXCH; ++it) M[it] = lane_max(dense_absmax8(X[it], selbits, slot_any, it), 6);
        chunk_tree_max<MAXCH>(M, A.cpg_q);
    }

    uint16_t* scale_row = reinterpret_cast<uint16_t*>(A.wire + A.off_scale) + (uint64_t)row * (uint64_t)(d / A.gq);
    uint8_t* code_row = A.wire + A.off_codes + (uint64_t)row * (uint64_t)d * BITS / 8u;
    const bool dword3 = (d % 32) == 0;
    const int lanes_pg_q = A.gq >= kChunk ? kWave : A.gq / 8;
#pragma unroll
    for (int it = 0; it < MAXCH; ++it) {
        if (it < nch) {
        const int c0 = it * kChunk + (int)lane * 8;
        const bool act = c0 < d;
        const int grp = c0 / A.gq;
        const float m = A.cpg_q > 1 ? M[it] : lane_max(dense_absmax8(X[it], selbits, slot_any, it), A.lane_lv_q);
        uint32_t sh;
        if (A.fixed) {
            sh = step_roundup(act ? A.steps[grp] : 1.0f);
        } else {
            sh = m == 0.0f ? 0u : scale_roundup(m, q);
            const bool first = (A.gq >= kChunk) ? (lane == 0 && (it % A.cpg_q) == 0) : ((int)lane % lanes_pg_q == 0);
            if (first && act) scale_row[grp] = (uint16_t)sh;
        }
        const float s = f16_value(sh);
        const float inv = sh ? __builtin_amdgcn_rcpf(s) : 0.0f;
        const float a = f16_value(CF[it] & 0xFFFFu), b0 = f16_value(CF[it] >> 16);
        float r[8];
        widen8(RV[it], r);
        // a6-a8: quantize, pack, reconstruct
        Packed<BITS> pk{};
        float H[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float e = X[it][j];
            const bool slot_has = slot_any.test(it * 8 + j);
            bool is_out = false;
            if (slot_has) {
                is_out = selbits.test(it * 8 + j);
                if (is_out) e = 0.0f;
            }
            float tc = __builtin_amdgcn_fmed3f(e * inv, -q, q);
            float mg = tc + kMagic;
            float qf = mg - kMagic;
            if (__builtin_fabsf(tc - qf) > kNearHalf) {
                tc = __builtin_amdgcn_fmed3f(e / s, -q, q);
                mg = tc + kMagic;
                qf = mg - kMagic;
            }
            pack_put<BITS>(pk, j, __float_as_uint(mg));
            float eh = qf * s;
            if (slot_has && is_out) eh = f16_value(f16_rne_sat(X[it][j]));
            H[j] = (a * r[j] + b0) + eh;
        }
        store_codes<BITS>(code_row, it, lane, act, dword3, pk);
        if (A.xhat && act) store_xhat(A, rbase + c0, H);
        }
    }
}

// ---------------------------------------------------------------------------
// Decode / reconstruct: one wavefront per token row, pure streaming.

template <int BITS, int MAXCH>
__global__ __launch_bounds__(kBlock) void rac_decode_kernel(Args A) {
    __shared__ uint32_t s_ent_all[kWavesPerBlock][kWave];
    const uint32_t lane = threadIdx.x & (kWave - 1);
    const uint32_t wv = threadIdx.x / kWave;
    const int64_t row = (int64_t)blockIdx.x * kWavesPerBlock + wv;
    if (row >= A.tokens) return;
    const int d = A.d, nch = A.nch, k = A.k;
    const uint64_t rbase = (uint64_t)row * (uint64_t)d;
    uint32_t* s_ent = s_ent_all[wv];

    // outliers of this row: owner lanes mark their slots
    SlotMask<MAXCH> selbits{}, slot_any{};
    if (k > 0) {
        const uint32_t* ol = reinterpret_cast<const uint32_t*>(A.wire + A.off_outl) + (uint64_t)row * (uint64_t)k;
        const uint32_t ent = lane < (uint32_t)k ? ol[lane] : 0u;
        s_ent[lane] = ent;
        wave_lds_sync();
        for (int i = 0; i < k; ++i) {
            const uint32_t c = rdlane(ent, i) & 0xFFFFu;
            if (c < (uint32_t)d) {
                const uint32_t owner = (c % kChunk) / 8u;
                const int slot = (int)((c / kChunk) * 8u + (c % 8u));
                slot_any.set(slot);
                if (lane == owner) selbits.set(slot);
            }
        }
    }

    const uint32_t* coef_row = reinterpret_cast<const uint32_t*>(A.wire + A.off_coef) + (uint64_t)row * (uint64_t)(d / A.ga);
    const uint16_t* scale_row = reinterpret_cast<const uint16_t*>(A.wire + A.off_scale) + (uint64_t)row * (uint64_t)(d / A.gq);
    const uint8_t* code_row = A.wire + A.off_codes + (uint64_t)row * (uint64_t)d * BITS / 8u;
    const bool dword3 = (d % 32) == 0;
#pragma unroll
    for (int it = 0; it < MAXCH; ++it) {
        if (it < nch) {
        const int c0 = it * kChunk + (int)lane * 8;
        const bool act = c0 < d;
        uint4 rv = make_uint4(0, 0, 0, 0);
        uint32_t cf = 0, sh = 0, lo, hi;
        if (act) {
            if (A.ref) rv = *reinterpret_cast<const uint4*>(A.ref + rbase + c0);
            cf = coef_row[c0 / A.ga];
            sh = A.fixed ? step_roundup(A.steps[c0 / A.gq]) : (uint32_t)scale_row[c0 / A.gq];
        }
        load_codes<BITS>(code_row, it, lane, act, dword3, lo, hi);
        const float a = f16_value(cf & 0xFFFFu), b0 = f16_value(cf >> 16);
        const float s = f16_value(sh);
        const float r[8] = {bf16_lo(rv.x), bf16_hi(rv.x), bf16_lo(rv.y), bf16_hi(rv.y),
                            bf16_lo(rv.z), bf16_hi(rv.z), bf16_lo(rv.w), bf16_hi(rv.w)};
        float H[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float eh = (float)code_at<BITS>(lo, hi, j) * s;
            if (slot_any.test(it * 8 + j)) {
                if (selbits.test(it * 8 + j)) {
                    const uint32_t c = (uint32_t)c0 + (uint32_t)j;
                    for (int i = 0; i < k; ++i)
                        if ((s_ent[i] & 0xFFFFu) == c) eh = f16_value(s_ent[i] >> 16);
                }
            }
            const float rt = a * r[j] + b0;
            H[j] = rt + eh;
        }
        if (act) store_xhat(A, rbase + c0, H);
        }
    }
}

// ---------------------------------------------------------------------------
// Host side

bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }
int ilog2(int64_t v) { int l = 0; while ((int64_t(1) << l) < v) ++l; return l; }
uint64_t up256(uint64_t v) { return (v + 255u) & ~uint64_t(255); }

bool config_valid(const rac_config* c) {
    if (!c) return false;
    if (c->tokens < 0 || c->tokens > 0xFFFFFFFFll) return false;
    if (c->hidden < 8 || c->hidden > 65535 || c->hidden % 8 != 0) return false;
    if (!is_pow2(c->group_align) || c->group_align < 8 || c->group_align > c->hidden ||
        c->hidden % c->group_align != 0)
        return false;
    if (!is_pow2(c->group_quant) || c->group_quant < 8 || c->group_quant > c->hidden ||
        c->hidden % c->group_quant != 0)
        return false;
    if (c->bits != 2 && c->bits != 3 && c->bits != 4 && c->bits != 8) return false;
    if (c->outlier_k < 0 || c->outlier_k > 64 || c->outlier_k > c->hidden) return false;
    if (c->flags & ~uint32_t(RAC_FLAG_FIXED_STEP | RAC_FLAG_XHAT_BF16)) return false;
    return true;
}

struct Sizes {
    rac_layout L;
    uint64_t coef, scale, codes, outl;
};

Sizes sizes_of(const rac_config* c) {
    Sizes s;
    const uint64_t T = (uint64_t)c->tokens, d = (uint64_t)c->hidden;
    s.coef = T * (d / (uint64_t)c->group_align) * 4u;
    s.scale = (c->flags & RAC_FLAG_FIXED_STEP) ? 0u : T * (d / (uint64_t)c->group_quant) * 2u;
    s.codes = T * d * (uint64_t)c->bits / 8u;
    s.outl = T * (uint64_t)c->outlier_k * 4u;
    s.L.off_coef = 256;
    s.L.off_scale = up256(s.L.off_coef + s.coef);
    s.L.off_codes = up256(s.L.off_scale + s.scale);
    s.L.off_outl = up256(s.L.off_codes + s.codes);
    s.L.total = up256(s.L.off_outl + s.outl);
    return s;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

Args make_args(const rac_config* c, const Sizes& S) {
    Args A{};
    A.off_coef = S.L.off_coef;
    A.off_scale = S.L.off_scale;
    A.off_codes = S.L.off_codes;
    A.off_outl = S.L.off_outl;
    A.total = S.L.total;
    A.end_coef = S.L.off_coef + S.coef;
    A.end_scale = S.L.off_scale + S.scale;
    A.end_codes = S.L.off_codes + S.codes;
    A.end_outl = S.L.off_outl + S.outl;
    A.tokens = c->tokens;
    A.d = c->hidden;
    A.nch = (c->hidden + kChunk - 1) / kChunk;
    A.ga = c->group_align;
    A.gq = c->group_quant;
    A.lane_lv_a = ilog2(c->group_align >= kChunk ? kChunk / 8 : c->group_align / 8);
    A.lane_lv_q = ilog2(c->group_quant >= kChunk ? kChunk / 8 : c->group_quant / 8);
    A.cpg_a = c->group_align >= kChunk ? c->group_align / kChunk : 1;
    A.cpg_q = c->group_quant >= kChunk ? c->group_quant / kChunk : 1;
    A.k = c->outlier_k;
    A.fixed = (c->flags & RAC_FLAG_FIXED_STEP) ? 1 : 0;
    A.xhat_bf16 = (c->flags & RAC_FLAG_XHAT_BF16) ? 1 : 0;
    return A;
}

void fill_header(Args& A, const rac_config* c, bool zero_ref) {
    uint8_t h[96] = {0};
    auto put16 = [&](int o, uint32_t v) { h[o] = (uint8_t)v; h[o + 1] = (uint8_t)(v >> 8); };
    auto put32 = [&](int o, uint32_t v) { for (int i = 0; i < 4; ++i) h[o + i] = (uint8_t)(v >> (8 * i)); };
    auto put64 = [&](int o, uint64_t v) { for (int i = 0; i < 8; ++i) h[o + i] = (uint8_t)(v >> (8 * i)); };
    uint32_t flags = 0;
    if (c->outlier_k > 0) flags |= 1u;
    if (c->flags & RAC_FLAG_FIXED_STEP) flags |= 2u;
    if (zero_ref) flags |= 4u;
    put32(0, 0x31434152u);
    put16(4, 1u);
    put16(6, flags);
    put32(8, (uint32_t)c->tokens);
    put32(12, (uint32_t)c->hidden);
    put32(16, (uint32_t)c->group_align);
    put32(20, (uint32_t)c->group_quant);
    h[24] = (uint8_t)c->bits;
    h[25] = 1;
    h[26] = (c->flags & RAC_FLAG_FIXED_STEP) ? 0 : 1;
    h[27] = c->outlier_k > 0 ? 1 : 0;
    put16(28, (uint32_t)c->outlier_k);
    put64(32, A.off_coef);
    put64(40, A.off_scale);
    put64(48, A.off_codes);
    put64(56, A.off_outl);
    put64(64, A.total);
    for (int i = 0; i < 24; ++i)
        A.hdr[i] = (uint32_t)h[4 * i] | ((uint32_t)h[4 * i + 1] << 8) | ((uint32_t)h[4 * i + 2] << 16) |
                   ((uint32_t)h[4 * i + 3] << 24);
}

using KernelFn = void (*)(Args);

template <int BITS, int MAXCH>
struct EncK { static constexpr KernelFn fn = rac_encode_kernel<BITS, MAXCH>; };
template <int BITS, int MAXCH>
struct DecK { static constexpr KernelFn fn = rac_decode_kernel<BITS, MAXCH>; };

template <template <int, int> class K>
KernelFn pick(int bits, int nch) {
    const bool small = nch <= 8;
    switch (bits) {
        case 2: return small ? K<2, 8>::fn : K<2, 16>::fn;
        case 3: return small ? K<3, 8>::fn : K<3, 16>::fn;
        case 4: return small ? K<4, 8>::fn : K<4, 16>::fn;
        default: return small ? K<8, 8>::fn : K<8, 16>::fn;
    }
}

rac_status launch(KernelFn fn, Args A, int64_t rows, hipStream_t stream) {
    const int64_t blocks = rows > 0 ? (rows + kWavesPerBlock - 1) / kWavesPerBlock : 1;
    void* args[] = {&A};
    const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(fn), dim3((unsigned)blocks),
                                         dim3(kBlock), args, 0, stream);
    return e == hipSuccess ? RAC_OK : RAC_ERR_HIP;
}

rac_status common_checks(const rac_config* cfg) {
    if (!config_valid(cfg)) return RAC_ERR_INVALID;
    if (cfg->hidden > 16 * kChunk) return RAC_ERR_UNSUPPORTED;
    return RAC_OK;
}

rac_status run_decode(const rac_config* cfg, const void* wire, const void* ref, const float* steps,
                      void* xhat, hipStream_t stream) {
    rac_status st = common_checks(cfg);
    if (st != RAC_OK) return st;
    if (!wire || (cfg->tokens > 0 && !xhat)) return RAC_ERR_INVALID;
    if ((cfg->flags & RAC_FLAG_FIXED_STEP) && !steps) return RAC_ERR_INVALID;
    if (!aligned(wire, 256) || !aligned(xhat, 16) || (ref && !aligned(ref, 16)) ||
        (steps && !aligned(steps, 4)))
        return RAC_ERR_ALIGN;
    if (cfg->tokens == 0) return RAC_OK;
    const Sizes S = sizes_of(cfg);
    Args A = make_args(cfg, S);
    A.wire = const_cast<uint8_t*>(static_cast<const uint8_t*>(wire));
    A.ref = static_cast<const uint16_t*>(ref);
    A.steps = steps;
    A.xhat = xhat;
    return launch(pick<DecK>(cfg->bits, A.nch), A, cfg->tokens, stream);
}

}  // namespace

extern "C" {

rac_status rac_wire_layout(const rac_config* cfg, rac_layout* out) {
    if (!config_valid(cfg) || !out) return RAC_ERR_INVALID;
    *out = sizes_of(cfg).L;
    return RAC_OK;
}

size_t rac_wire_size(const rac_config* cfg) {
    if (!config_valid(cfg)) return 0;
    return (size_t)sizes_of(cfg).L.total;
}

rac_status rac_parse_header(const void* header_host, size_t len, rac_config* out, int* zero_ref) {
    if (!header_host || !out) return RAC_ERR_INVALID;
    if (len < 256) return RAC_ERR_FORMAT;
    const uint8_t* h = static_cast<const uint8_t*>(header_host);
    auto g16 = [&](int o) { return (uint32_t)h[o] | ((uint32_t)h[o + 1] << 8); };
    auto g32 = [&](int o) { uint32_t v = 0; for (int i = 3; i >= 0; --i) v = (v << 8) | h[o + i]; return v; };
    auto g64 = [&](int o) { uint64_t v = 0; for (int i = 7; i >= 0; --i) v = (v << 8) | h[o + i]; return v; };
    if (g32(0) != 0x31434152u || g16(4) != 1u) return RAC_ERR_FORMAT;
    const uint32_t flags = g16(6);
    if (flags & ~7u) return RAC_ERR_FORMAT;
    rac_config c{};
    c.tokens = g32(8);
    c.hidden = (int32_t)g32(12);
    c.group_align = (int32_t)g32(16);
    c.group_quant = (int32_t)g32(20);
    c.bits = h[24];
    c.outlier_k = (int32_t)g16(28);
    c.flags = (flags & 2u) ? RAC_FLAG_FIXED_STEP : 0u;
    if (g32(12) > 65535u || g32(16) > 65535u || g32(20) > 65535u) return RAC_ERR_FORMAT;
    if (!config_valid(&c)) return RAC_ERR_FORMAT;
    if (((flags & 1u) != 0) != (c.outlier_k > 0)) return RAC_ERR_FORMAT;
    if (h[25] != 1 || h[26] != ((flags & 2u) ? 0 : 1) || h[27] != (c.outlier_k > 0 ? 1 : 0))
        return RAC_ERR_FORMAT;
    const Sizes S = sizes_of(&c);
    if (g64(32) != S.L.off_coef || g64(40) != S.L.off_scale || g64(48) != S.L.off_codes ||
        g64(56) != S.L.off_outl || g64(64) != S.L.total)
        return RAC_ERR_FORMAT;
    for (int i = 30; i < 32; ++i)
        if (h[i]) return RAC_ERR_FORMAT;
    for (int i = 72; i < 256; ++i)
        if (h[i]) return RAC_ERR_FORMAT;
    *out = c;
    if (zero_ref) *zero_ref = (flags & 4u) ? 1 : 0;
    return RAC_OK;
}

rac_status rac_encode(const rac_config* cfg, const void* x, const void* ref, const float* fixed_steps,
                      void* wire, size_t wire_cap, void* xhat, rac_stream_t stream) {
    rac_status st = common_checks(cfg);
    if (st != RAC_OK) return st;
    if (!wire || (cfg->tokens > 0 && !x)) return RAC_ERR_INVALID;
    if ((cfg->flags & RAC_FLAG_FIXED_STEP) && !fixed_steps) return RAC_ERR_INVALID;
    if (!aligned(wire, 256) || !aligned(x, 16) || (ref && !aligned(ref, 16)) ||
        (xhat && !aligned(xhat, 16)) || (fixed_steps && !aligned(fixed_steps, 4)))
        return RAC_ERR_ALIGN;
    const Sizes S = sizes_of(cfg);
    if (wire_cap < S.L.total) return RAC_ERR_CAPACITY;
    Args A = make_args(cfg, S);
    A.x = static_cast<const uint16_t*>(x);
    A.ref = static_cast<const uint16_t*>(ref);
    A.steps = (cfg->flags & RAC_FLAG_FIXED_STEP) ? fixed_steps : nullptr;
    A.wire = static_cast<uint8_t*>(wire);
    A.xhat = xhat;
    A.write_header = 1;
    fill_header(A, cfg, ref == nullptr);
    return launch(pick<EncK>(cfg->bits, A.nch), A, cfg->tokens, stream);
}

rac_status rac_reconstruct(const rac_config* cfg, const void* wire, const void* ref,
                           const float* fixed_steps, void* xhat, rac_stream_t stream) {
    return run_decode(cfg, wire, ref, fixed_steps, xhat, stream);
}

rac_status rac_decode(const rac_config* cfg, const void* wire, const void* ref, const float* fixed_steps,
                      void* xhat, rac_stream_t stream) {
    return run_decode(cfg, wire, ref, fixed_steps, xhat, stream);
}

const char* rac_status_string(rac_status s) {
    switch (s) {
        case RAC_OK: return "ok";
        case RAC_ERR_INVALID: return "invalid argument";
        case RAC_ERR_ALIGN: return "misaligned pointer";
        case RAC_ERR_CAPACITY: return "wire buffer too small";
        case RAC_ERR_HIP: return "HIP kernel launch failed";
        case RAC_ERR_FORMAT: return "malformed wire header";
        case RAC_ERR_UNSUPPORTED: return "configuration not supported by the kernels";
    }
    return "unknown status";
}

}  // extern "C"
