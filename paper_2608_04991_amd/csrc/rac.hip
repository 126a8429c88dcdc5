// rac.hip - gfx950 kernels and C ABI of the RAC aligned residual codec.
//
// Method: the paper's Section "Quality- and Cost-Constrained Aligned Residual
// Encoding" (Eq. affine-fit, Eq. aligned-residual, Eq. residual-quantization,
// the outlier paragraph, Eq. residual-reconstruction).  The contract of every
// entry point is documented in include/rac.h.
//
// Mapping onto CDNA4.  The codec is a per-token-row stream with no dense
// contraction, so it is HBM-bound and uses no MFMA.  One workgroup owns one
// token row and one 64-lane wavefront owns one 512-channel chunk of it: lane l
// of wave w holds channels [512w + 8l, 512w + 8l + 8), one 128-bit load of x
// and one of ref per lane, fully coalesced.  Each lane keeps its 8 channels in
// registers through fit, residual, outlier choice, scale, quantization,
// packing and the fused sender reconstruction, so every byte of x/ref is read
// from HBM once and every output byte written once.  Work that spans chunks
// (the per-token outlier choice, groups wider than 512 channels) goes through
// LDS with workgroup barriers; everything else is wave-local.  (The
// per-token outlier encode deals a row's chunks round four wavefronts, two or
// four chunks each.)  Up to a few rows per resident workgroup the grid is the
// resident workgroups, taking rows in strides with the next row prefetched;
// beyond that, one workgroup per row, which keeps the rows in flight close
// together in memory.
//
// Exactness.  The sums of the fit follow a fixed pairwise tree over channel
// order: a lane-local tree over its 8 contiguous channels, a butterfly across
// lanes whose every step adds the partial sums of two adjacent aligned blocks
// (DPP quad_perm / row_half_mirror / row_mirror, then v_permlane16_swap and
// v_permlane32_swap), then a pairwise tree over chunks.  Floating-point
// addition is commutative, so that reproduces the canonical pairwise sum
// exactly.  The file is compiled with -ffp-contract=off so no multiply-add is
// fused, and divisions stay correctly rounded.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <mutex>

#include "rac.h"

namespace {

constexpr int kWave = 64;
constexpr int kChunk = 512;       // channels per wavefront (8 per lane)
constexpr int kMaxWaves = 16;     // rows up to 8192 channels
constexpr int kCandCap = 64;      // outlier candidates ranked by one wavefront (twice that for k > 48)
constexpr int kMaxGatherRows = 64; // rows per workgroup with a gathered reference
constexpr int kStridedRowsMax = 6; // beyond this many rows per resident workgroup: one workgroup per row
constexpr uint32_t kMaxDispatchItems = 0xFFFFFFFFu;  // work-items one dispatch holds (per dimension)
constexpr float kMagic = 12582912.0f;  // 1.5 * 2^23: adding it rounds to an integer (RNE)
// Quotients t' = E * (1/s) within this distance of a half-integer are
// recomputed with the correctly rounded division E / s.  |t' - E/s| is below
// 2 ulp(128) = 2^-16 for |t'| <= 128, so the fast rounding is exact elsewhere.
constexpr float kNearHalf = 0.5f - 0x1p-14f;

struct alignas(8) Args {
    // hot-path fields
    const uint16_t* x;
    const uint16_t* ref;      // the reference, or with ref_rows the store its rows come from
    const int32_t* ref_rows;  // per token row: the store row of its reference (NULL: row t of ref)
    uint32_t store_rows;
    const float* steps;
    uint32_t* coef;     // wire sections
    uint16_t* scale;
    uint8_t* codes;
    uint32_t* outl;     // per-token outliers, or the fp16 values of per-group ones
    uint16_t* gval;     // per-group outliers: fp16 values [T][d/g_q][k_g] (= outl)
    uint8_t* goff;      //                     u8 in-group offsets [T][d/g_q][k_g]
    void* xhat;
    uint32_t tokens;    // < 2^31, so row + gridDim.x never wraps
    int32_t d;
    int32_t code_row_bytes;  // d * bits / 8
    int32_t nch;        // 512-channel chunks per row = wavefronts per workgroup
    int32_t lg_a, lg_q; // log2 of the group sizes
    int32_t lane_lv_a;  // butterfly levels inside a chunk: log2(min(g, 512) / 8)
    int32_t lane_lv_q;
    int32_t lg_cpg_a;   // log2 chunks per group (0 when a group fits in a chunk)
    int32_t lg_cpg_q;
    int32_t k;          // outliers per row, or per group with gout
    int32_t gout;       // per-group outlier mode
    int32_t cf_given;   // pooled fit: the pairs are given (see pool_first_rows)
    int32_t segments;   // pooled fit: segment count and row starts [segments + 1]
    const int32_t* seg_start;
    int32_t pool_first_rows;  // pooled fit: a segment's pair is in its first row only
    int32_t fixed;
    int32_t xhat_bf16;
    float inv_ga;       // 1 / g_a (exact, power of two)
    int32_t launch_shape;  // (read by the host only) 0 by rows per workgroup, 1 strided, 2 one workgroup per row
    // header and padding (written once, by the first wavefront)
    int32_t write_header;
    uint8_t* wire;
    uint64_t off_scale, off_codes, off_outl, off_ooff, total;
    uint64_t end_coef, end_scale, end_codes, end_outl, end_ooff;  // first byte after each section
    uint32_t hdr[24];   // first 96 bytes of the header; the rest is zero
};

// ---------------------------------------------------------------------------
// Raw buffer access.  Each row section (x, ref, coef, scale, codes, outliers,
// xhat of one token row) is addressed through a buffer resource whose range is
// exactly that section; the hardware drops a store at an offset outside the
// range and returns 0 for such a load.  Lanes without work (the tail of a
// partial chunk, lanes that do not own a group's coefficient) take an offset
// outside the range instead of a branch, so every store of a row is issued
// unconditionally and the wait for the next row's prefetched loads does not
// have to wait for this row's stores as well.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr uint32_t kOut = 0x80000000u;       // an offset outside every range
constexpr int kRawBufferWord3 = 0x00020000;  // untyped buffer, 32-bit data format field
// s_waitcnt operand: vector memory count 0, export and LDS/scalar counts left
// at their maxima (no wait on them)
constexpr int kWaitVmem0 = 0x0F70;

// Resource for `bytes` bytes at element `i` of array `p`.  The address is
// formed in integer arithmetic: p may be null when the range is empty.
template <class T>
__device__ __forceinline__ Rsrc rsrc(const T* p, uint64_t i, uint32_t bytes) {
    const uint64_t a = (uint64_t)(uintptr_t)p + i * sizeof(T);
    return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(a), (short)0, (int)bytes, kRawBufferWord3);
}
__device__ __forceinline__ uint4 bload128(Rsrc r, uint32_t off) {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint2 bload64(Rsrc r, uint32_t off) {
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0);
    return make_uint2(v.x, v.y);
}
__device__ __forceinline__ uint32_t bload32(Rsrc r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
}
__device__ __forceinline__ uint32_t bload16(Rsrc r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0);
}
__device__ __forceinline__ uint32_t bload8(Rsrc r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b8(r, (int)off, 0, 0);
}
// The 128-bit stores (the reconstruction, 1 KiB per wavefront instruction)
// and the code stores (whole cache lines per wavefront) are streaming: written
// once and not read again by the kernel, they carry the non-temporal hint, so
// they do not displace lines in the caches.  Measured on back-to-back encodes
// of 65536 x 3584: 412 -> 397 us, and 4096 x 4096: 32.1 -> 29.5 us.  The
// narrow per-row fields (coefficients, scales, outliers) keep the default
// policy: rows of 112 or 56 bytes share cache lines with their neighbours,
// and non-temporal partial lines measured 4% slower.
constexpr int kStream = 2;  // cache-policy operand of the buffer store: non-temporal

__device__ __forceinline__ void bstore128(Rsrc r, uint32_t off, uint4 v) {
    __builtin_amdgcn_raw_buffer_store_b128((u32x4){v.x, v.y, v.z, v.w}, r, (int)off, 0, kStream);
}
__device__ __forceinline__ void sstore64(Rsrc r, uint32_t off, uint32_t lo, uint32_t hi) {
    __builtin_amdgcn_raw_buffer_store_b64((u32x2){lo, hi}, r, (int)off, 0, kStream);
}
__device__ __forceinline__ void sstore32(Rsrc r, uint32_t off, uint32_t v) {
    __builtin_amdgcn_raw_buffer_store_b32(v, r, (int)off, 0, kStream);
}
__device__ __forceinline__ void sstore16(Rsrc r, uint32_t off, uint32_t v) {
    __builtin_amdgcn_raw_buffer_store_b16((uint16_t)v, r, (int)off, 0, kStream);
}
__device__ __forceinline__ void bstore64(Rsrc r, uint32_t off, uint32_t lo, uint32_t hi) {
    __builtin_amdgcn_raw_buffer_store_b64((u32x2){lo, hi}, r, (int)off, 0, 0);
}
__device__ __forceinline__ void bstore32(Rsrc r, uint32_t off, uint32_t v) {
    __builtin_amdgcn_raw_buffer_store_b32(v, r, (int)off, 0, 0);
}
__device__ __forceinline__ void bstore16(Rsrc r, uint32_t off, uint32_t v) {
    __builtin_amdgcn_raw_buffer_store_b16((uint16_t)v, r, (int)off, 0, 0);
}
__device__ __forceinline__ void bstore8(Rsrc r, uint32_t off, uint32_t v) {
    __builtin_amdgcn_raw_buffer_store_b8((uint8_t)v, r, (int)off, 0, 0);
}

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

// The fp16 fields of the wire (alpha, beta, scale, outlier values) hold the
// IEEE result of their rounding: a magnitude whose round-to-nearest-even
// overflows is +-infinity, and a scale with no finite fp16 covering the
// group is +infinity.  That reports the saturation in the wire at no cost;
// both ends compute with +-65504 in its place.
__device__ __forceinline__ uint32_t f16_rne(float v) {
    const _Float16 h = (_Float16)v;
    return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

// The value a wire fp16 field stands for: +-infinity reads as +-65504.
__device__ __forceinline__ float f16_wire(uint32_t bits) {
    return __builtin_fminf(__builtin_fmaxf(f16_value(bits), -65504.0f), 65504.0f);
}

// fp32 -> bf16 pattern, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t bf16_rne(float v) {
    const uint32_t u = __float_as_uint(v);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Smallest positive fp16 h with value(h) * q >= m  (m > 0); +infinity
// (0x7C00, read as 65504, the codes then clip) if no finite fp16 is.
// value(h) * q is exact in binary32, so the test below is an exact
// comparison.  y = m * fl(1/q) is within 2^-23 (relative) of m/q, so its RNE
// fp16 rounding h0 is either the answer or one step below it: if value(h0)
// >= m/q, then y was at least the midpoint below h0 and value(h0-1) < m/q; if
// value(h0) < m/q, then y was at most the midpoint above h0 and
// value(h0+1) >= m/q.
__device__ __forceinline__ uint32_t scale_roundup(float m, float q, float inv_q) {
    uint32_t h = f16_rne_sat(m * inv_q);
    h = h < 1u ? 1u : h;
    h = f16_value(h) * q >= m ? h : h + 1u;
    return m > 65504.0f * q ? 0x7C00u : h;
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
// gives (0, m_x).  Returns the fp16 pair (alpha | beta << 16), each the IEEE
// rounding (+-infinity past the fp16 range).
__device__ __forceinline__ uint32_t fit_coef(float crr, float crx, float mr, float mx) {
    const bool flat = crr == 0.0f;
    const float as = flat ? 0.0f : crx / crr;
    const float bs = flat ? mx : mx - as * mr;
    return f16_rne(as) | (f16_rne(bs) << 16);
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

// Same with a compile-time depth (LV >= 0); LV < 0 falls back to `levels`.
template <int LV>
__device__ __forceinline__ float lsum(float v, int levels) {
    if constexpr (LV < 0) {
        return lane_sum(v, levels);
    } else {
        if constexpr (LV > 0) v = v + dpp<0xB1>(v);
        if constexpr (LV > 1) v = v + dpp<0x4E>(v);
        if constexpr (LV > 2) v = v + dpp<0x141>(v);
        if constexpr (LV > 3) v = v + dpp<0x140>(v);
        if constexpr (LV > 4) v = pair16_sum(v);
        if constexpr (LV > 5) v = pair32_sum(v);
        return v;
    }
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

// Max over the lanes of an aligned block of non-negative, non-NaN values: on
// such values the unsigned order of the bit patterns is the float order, and
// an integer max folds into one DPP instruction per level.
template <int LV>
__device__ __forceinline__ float lmax(float f, int levels) {
    if constexpr (LV < 0) {
        return lane_max(f, levels);
    } else {
        uint32_t v = __float_as_uint(f);
        if constexpr (LV > 0) v = __builtin_elementwise_max(v, dpp_u<0xB1>(v));
        if constexpr (LV > 1) v = __builtin_elementwise_max(v, dpp_u<0x4E>(v));
        if constexpr (LV > 2) v = __builtin_elementwise_max(v, dpp_u<0x141>(v));
        if constexpr (LV > 3) v = __builtin_elementwise_max(v, dpp_u<0x140>(v));
        if constexpr (LV > 4) {
            auto p = __builtin_amdgcn_permlane16_swap((int)v, (int)v, false, false);
            v = __builtin_elementwise_max((uint32_t)p[0], (uint32_t)p[1]);
        }
        if constexpr (LV > 5) {
            auto p = __builtin_amdgcn_permlane32_swap((int)v, (int)v, false, false);
            v = __builtin_elementwise_max((uint32_t)p[0], (uint32_t)p[1]);
        }
        return __uint_as_float(v);
    }
}

__device__ __forceinline__ float tree8(const float* v) {
    return ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
}

__device__ __forceinline__ uint32_t mbcnt64(uint64_t m) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }

// A value known to be equal in all lanes, moved to a scalar register.
__device__ __forceinline__ uint32_t uniform(uint32_t v) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)v); }

__device__ __forceinline__ uint32_t rdlane(uint32_t v, int l) {
    return (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}

// Orders this wavefront's LDS writes before its later LDS reads by other
// lanes (LDS executes one wavefront's instructions in order; this keeps the
// compiler from reordering them).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

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
    zero_bytes(A.wire, A.end_outl, A.off_ooff, lane);
    zero_bytes(A.wire, A.end_ooff, A.total, lane);
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

// Codes of 8 channels from their rounding patterns t + 1.5 * 2^23, whose
// low bits are the two's-complement code: each funnel shift moves the codes
// gathered so far down by BITS and puts the next one on top.
template <int BITS>
__device__ __forceinline__ Packed<BITS> pack8(const float* mg) {
    Packed<BITS> p{};
    if constexpr (BITS == 8) {
#pragma unroll
        for (int j = 0; j < 4; ++j) p.lo = __builtin_amdgcn_alignbit(__float_as_uint(mg[j]), p.lo, 8u);
#pragma unroll
        for (int j = 4; j < 8; ++j) p.hi = __builtin_amdgcn_alignbit(__float_as_uint(mg[j]), p.hi, 8u);
    } else {
        uint32_t w = 0u;
#pragma unroll
        for (int j = 0; j < 8; ++j) w = __builtin_amdgcn_alignbit(__float_as_uint(mg[j]), w, (uint32_t)BITS);
        p.w = w >> (32 - 8 * BITS);
    }
    return p;
}

// Store the packed codes of chunk `it` for this lane into the row's code
// section `rc`.  Lane l's 8 channels occupy bytes [l*BITS, l*BITS + BITS) of
// the chunk's 64*BITS bytes; lanes past the end of the row fall outside the
// section's range.
template <int BITS>
__device__ __forceinline__ void store_codes(Rsrc rc, int it, uint32_t lane, bool dword_ok, const Packed<BITS>& p);

template <>
__device__ __forceinline__ void store_codes<2>(Rsrc rc, int it, uint32_t lane, bool, const Packed<2>& p) {
    sstore16(rc, (uint32_t)it * 128u + lane * 2u, p.w);
}
template <>
__device__ __forceinline__ void store_codes<4>(Rsrc rc, int it, uint32_t lane, bool, const Packed<4>& p) {
    sstore32(rc, (uint32_t)it * 256u + lane * 4u, p.w);
}
template <>
__device__ __forceinline__ void store_codes<8>(Rsrc rc, int it, uint32_t lane, bool, const Packed<8>& p) {
    sstore64(rc, (uint32_t)it * 512u + lane * 8u, p.lo, p.hi);
}
template <>
__device__ __forceinline__ void store_codes<3>(Rsrc rc, int it, uint32_t lane, bool dword_ok, const Packed<3>& p) {
    // Four lanes own 96 contiguous bits = 3 dwords; lane j of the quad writes
    // dword j from its own 24 bits and the next lane's.  Rows whose length is
    // not a multiple of 32 channels are written bytewise.
    const uint32_t base = (uint32_t)it * 192u;
    if (dword_ok) {
        const uint32_t nxt = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)p.w, 0x39 /* quad_perm [1,2,3,0] */,
                                                                   0xF, 0xF, false);
        const uint32_t j = lane & 3u;
        const uint32_t dw = j == 0 ? (p.w | (nxt << 24))
                          : j == 1 ? ((p.w >> 8) | (nxt << 16))
                                   : ((p.w >> 16) | (nxt << 8));
        sstore32(rc, j < 3u ? base + ((lane >> 2) * 3u + j) * 4u : kOut, dw);
    } else {
        bstore8(rc, base + lane * 3u + 0u, p.w);
        bstore8(rc, base + lane * 3u + 1u, p.w >> 8);
        bstore8(rc, base + lane * 3u + 2u, p.w >> 16);
    }
}

// Load this lane's packed codes of chunk `it` from the row's code section
// (inverse of store_codes; lanes past the end of the row read zeros).
template <int BITS>
__device__ __forceinline__ void load_codes(Rsrc rc, int it, uint32_t lane, bool dword_ok, uint32_t& lo,
                                           uint32_t& hi) {
    lo = hi = 0;
    if constexpr (BITS == 2) {
        lo = bload16(rc, (uint32_t)it * 128u + lane * 2u);
    } else if constexpr (BITS == 4) {
        lo = bload32(rc, (uint32_t)it * 256u + lane * 4u);
    } else if constexpr (BITS == 8) {
        const uint2 v = bload64(rc, (uint32_t)it * 512u + lane * 8u);
        lo = v.x;
        hi = v.y;
    } else {
        const uint32_t base = (uint32_t)it * 192u;
        if (dword_ok) {
            // lane j's 24 bits start at bit 24j of the quad's 96 bits
            const uint32_t j = lane & 3u;
            const uint32_t q0 = base + (lane >> 2) * 12u;
            const uint32_t i0 = (24u * j) >> 5;
            const uint32_t w0 = bload32(rc, q0 + i0 * 4u);
            const uint32_t w1 = bload32(rc, j == 3u ? kOut : q0 + (i0 + 1u) * 4u);
            const uint32_t sh = (24u * j) & 31u;
            lo = (sh ? ((w0 >> sh) | (w1 << (32u - sh))) : w0) & 0xFFFFFFu;
        } else {
            lo = bload8(rc, base + lane * 3u) | (bload8(rc, base + lane * 3u + 1u) << 8) |
                 (bload8(rc, base + lane * 3u + 2u) << 16);
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

// Pairwise tree over n (a power of two, <= 16) consecutive chunk partials.
__device__ __forceinline__ float tree_n(const float* p, int n) {
    float v[kMaxWaves];
#pragma unroll
    for (int i = 0; i < kMaxWaves; ++i) v[i] = i < n ? p[i] : 0.0f;
#pragma unroll
    for (int lv = 0; lv < 4; ++lv) {
        const int w = 1 << lv;
        if (w < n) {
#pragma unroll
            for (int i = 0; i + w < kMaxWaves; i += 2 * w) v[i] = v[i] + v[i + w];
        }
    }
    return v[0];
}

__device__ __forceinline__ float max_n(const float* p, int n) {
    float m = 0.0f;
    for (int i = 0; i < n; ++i) m = __builtin_fmaxf(m, p[i]);
    return m;
}

// Store this lane's 8 reconstructed channels at element offset c0 of the
// row's xhat section (fp32, or bf16 when bf16 is set).  Both forms issue two
// stores (the bf16 form's second one outside the range), so the number of
// stores per row does not depend on the format.
__device__ __forceinline__ void store_xhat(Rsrc rx, bool bf16, uint32_t c0, const float* H) {
    uint4 v0, v1;
    uint32_t o0, o1;
    if (bf16) {
        v0.x = bf16_rne(H[0]) | (bf16_rne(H[1]) << 16);
        v0.y = bf16_rne(H[2]) | (bf16_rne(H[3]) << 16);
        v0.z = bf16_rne(H[4]) | (bf16_rne(H[5]) << 16);
        v0.w = bf16_rne(H[6]) | (bf16_rne(H[7]) << 16);
        v1 = v0;
        o0 = c0 * 2u;
        o1 = kOut;
    } else {
        v0 = make_uint4(__float_as_uint(H[0]), __float_as_uint(H[1]), __float_as_uint(H[2]), __float_as_uint(H[3]));
        v1 = make_uint4(__float_as_uint(H[4]), __float_as_uint(H[5]), __float_as_uint(H[6]), __float_as_uint(H[7]));
        o0 = c0 * 4u;
        o1 = c0 * 4u + 16u;
    }
    bstore128(rx, o0, v0);
    bstore128(rx, o1, v1);
}

// A wavefront's LDS slice of one 512-channel chunk: lane l's channels
// 8l..8l+3 at float4 l and 8l+4..8l+7 at float4 kPlane + l.  Each access
// by the 64 lanes covers 1 KiB of consecutive float4s, and the 8-float4 gap
// puts the two planes in different banks for the transposed read below.
constexpr int kPlane = kWave + 8;
constexpr int kSlice = 2 * kPlane;  // float4 per slice

__device__ __forceinline__ void put8(float4* st, uint32_t lane, const float* v) {
    st[lane] = make_float4(v[0], v[1], v[2], v[3]);
    st[kPlane + lane] = make_float4(v[4], v[5], v[6], v[7]);
}

__device__ __forceinline__ void get8(const float4* st, uint32_t lane, float* v) {
    const float4 a = st[lane], b = st[kPlane + lane];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// Float offset of chunk channel c in a slice.
__device__ __forceinline__ uint32_t slice_float(uint32_t c) {
    return ((c & 4u) ? 4u * kPlane : 0u) + ((c >> 3) << 2) + (c & 3u);
}

// Store a chunk's reconstruction staged in the wavefront's slice `st`.  For
// fp32, lane m stores channels 4m..4m+3 and 256+4m..256+4m+3, so that each
// store instruction writes 1 KiB of contiguous memory (two interleaved
// 16-byte halves per lane cost HBM efficiency); bf16 lanes store their own 8
// channels.  Channels past the row fall outside the section's range.
__device__ __forceinline__ void emit_xhat(Rsrc rx, bool bf16, uint32_t chunk0, uint32_t lane, float4* st) {
    if (bf16) {
        float H[8];
        get8(st, lane, H);
        wave_lds_sync();
        store_xhat(rx, true, chunk0 + lane * 8u, H);
        return;
    }
    const uint32_t t = (lane & 1u) * kPlane + (lane >> 1);
    const float4 lo = st[t], hi = st[t + 32u];
    wave_lds_sync();  // the slice is rewritten by the next chunk
    bstore128(rx, (chunk0 + lane * 4u) * 4u,
              make_uint4(__float_as_uint(lo.x), __float_as_uint(lo.y), __float_as_uint(lo.z), __float_as_uint(lo.w)));
    bstore128(rx, (chunk0 + 256u + lane * 4u) * 4u,
              make_uint4(__float_as_uint(hi.x), __float_as_uint(hi.y), __float_as_uint(hi.z), __float_as_uint(hi.w)));
}

// Same as emit_xhat without a branch on the format: both forms read two
// float4 of the slice and issue two stores (the bf16 form's second one outside
// the range), so the memory operations of a row do not depend on the format.
__device__ __forceinline__ void emit_xhat_flat(Rsrc rx, bool bf16, uint32_t chunk0, uint32_t lane, float4* st) {
    const uint32_t tt = (lane & 1u) * kPlane + (lane >> 1);
    const uint32_t t0 = bf16 ? lane : tt, t1 = bf16 ? kPlane + lane : tt + 32u;
    const float4 lo = st[t0], hi = st[t1];
    wave_lds_sync();  // the slice is rewritten by the next chunk
    const uint4 pk = make_uint4(bf16_rne(lo.x) | (bf16_rne(lo.y) << 16), bf16_rne(lo.z) | (bf16_rne(lo.w) << 16),
                                bf16_rne(hi.x) | (bf16_rne(hi.y) << 16), bf16_rne(hi.z) | (bf16_rne(hi.w) << 16));
    const uint4 f0 = make_uint4(__float_as_uint(lo.x), __float_as_uint(lo.y), __float_as_uint(lo.z), __float_as_uint(lo.w));
    const uint4 f1 = make_uint4(__float_as_uint(hi.x), __float_as_uint(hi.y), __float_as_uint(hi.z), __float_as_uint(hi.w));
    bstore128(rx, bf16 ? (chunk0 + lane * 8u) * 2u : (chunk0 + lane * 4u) * 4u, bf16 ? pk : f0);
    bstore128(rx, bf16 ? kOut : (chunk0 + 256u + lane * 4u) * 4u, f1);
}

// Stage and store the lane's 8 reconstructed channels (the lane's channels
// 8l..8l+7 of the chunk starting at `chunk0`).
__device__ __forceinline__ void store_xhat_t(Rsrc rx, bool bf16, uint32_t chunk0, uint32_t lane, float4* st,
                                             const float* H) {
    if (bf16) {
        store_xhat(rx, true, chunk0 + lane * 8u, H);
        return;
    }
    put8(st, lane, H);
    wave_lds_sync();
    emit_xhat(rx, false, chunk0, lane, st);
}

// Buffer resource of one row of the reconstruction (range 0 when no
// reconstruction is wanted, which drops its stores).
__device__ __forceinline__ Rsrc xhat_row(const Args& A, uint32_t row) {
    const uint32_t es = A.xhat_bf16 ? 2u : 4u;
    return rsrc(static_cast<const uint8_t*>(A.xhat), (uint64_t)row * (uint64_t)A.d * es,
                A.xhat ? (uint32_t)A.d * es : 0u);
}

// Store-row indices of the rows a workgroup takes.  With a gathered reference
// the launch gives every workgroup at most kMaxGatherRows rows, so all of
// them are loaded once, before the row loop (a load inside the loop would
// make the compiler's wait counts conservative for the prefetched rows).
// Each wavefront holds the indices in one register, lane i for the
// workgroup's row i (token row blockIdx.x + i * gridDim.x, -1 past the last
// token); reading one is a lane read, with no memory wait and no barrier.
__device__ __forceinline__ int32_t load_ref_rows_v(const Args& A, uint32_t lane) {
    const uint64_t r = (uint64_t)blockIdx.x + (uint64_t)lane * gridDim.x;
    return (A.ref_rows && r < A.tokens) ? A.ref_rows[r] : -1;
}

__device__ __forceinline__ int32_t ref_index_v(const Args& A, int32_t cache, uint32_t n) {
    return A.ref_rows ? __builtin_amdgcn_readlane(cache, (int)(n & (uint32_t)(kWave - 1))) : 0;
}

// The index of the workgroup's first row, read directly, so that the first
// row's loads need not wait for the register copy.  Read through the constant
// address space (the array is read-only for the whole launch): that makes it a
// scalar load, which is waited for apart from the vector loads, and the kernels
// issue it first, before any store or barrier.
__device__ __forceinline__ int32_t first_ref_index(const Args& A) {
    using cptr = const __attribute__((address_space(4))) int32_t*;
    return (A.ref_rows && blockIdx.x < A.tokens) ? ((cptr)A.ref_rows)[blockIdx.x] : 0;
}

// Buffer resource of token row `row`'s reference: row `row` of ref, or, with
// a row index array, store row `ix`.  A missing reference, a row past the
// last token (`in` false) and an index outside the store give an empty range,
// which reads as a zero reference row.
__device__ __forceinline__ Rsrc ref_row(const Args& A, uint32_t row, bool in, int32_t ix) {
    uint32_t r = row;
    bool ok = in && A.ref != nullptr;
    if (A.ref_rows) {
        ok = ok && ix >= 0 && (uint32_t)ix < A.store_rows;
        r = ok ? (uint32_t)ix : 0u;
    }
    return rsrc(A.ref, (uint64_t)r * (uint64_t)A.d, ok ? (uint32_t)A.d * 2u : 0u);
}

// Workgroup-shared state of one row.
struct alignas(16) RowShared {
    uint32_t smax[kWave];           // max |E| bits over lane l of every wave (threshold search)
    uint64_t ckey[kCandCap];        // candidate key: |E| bits << 32 | (0xFFFF - channel)
    uint32_t cval[kCandCap];        // candidate E bits
    uint32_t cnt[4];                // [0] candidate count, [1..3] rotating block counters
    float part[5][kMaxWaves];       // chunk partials of groups wider than one chunk
};

// Sum of v over the workgroup (one value per wavefront, from lane 0), through
// three rotating LDS counters so that consecutive calls need one barrier each.
__device__ __forceinline__ uint32_t block_sum(RowShared& S, uint32_t v, int& it) {
    const int slot = 1 + it % 3;
    if (threadIdx.x == 0) S.cnt[1 + (it + 1) % 3] = 0u;
    if ((threadIdx.x & (kWave - 1)) == 0) atomicAdd(&S.cnt[slot], v);
    __syncthreads();
    ++it;
    return S.cnt[slot];
}

__device__ __forceinline__ uint32_t count8(const float* e, bool act, float t) {
    uint32_t n = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) n += (uint32_t)__builtin_popcountll(ballot(act & (__builtin_fabsf(e[j]) >= t)));
    return n;
}

__device__ __forceinline__ uint64_t cand_key(uint32_t ebits, uint32_t ch) {
    return ((uint64_t)(ebits & 0x7FFFFFFFu) << 32) | (uint64_t)(0xFFFFu - ch);
}

__device__ __forceinline__ uint32_t key_channel(uint64_t key) { return 0xFFFFu - (uint32_t)(key & 0xFFFFu); }

__device__ __forceinline__ uint64_t rdlane64(uint64_t v, int l) {
    return ((uint64_t)rdlane((uint32_t)(v >> 32), l) << 32) | (uint64_t)rdlane((uint32_t)v, l);
}

// Append this lane's elements satisfying p[j] to the LDS candidate list
// (one LDS atomic per wavefront reserves the slots).
__device__ __forceinline__ void append8(RowShared& S, uint32_t* counter, const float* e, const bool* p,
                                        int c0, uint32_t lane) {
    uint32_t n = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) n += (uint32_t)__builtin_popcountll(ballot(p[j]));
    if (!n) return;
    uint32_t base = 0u;
    if (lane == 0u) base = atomicAdd(counter, n);
    base = (uint32_t)__builtin_amdgcn_readfirstlane((int)base);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint64_t m = ballot(p[j]);
        if (m) {
            const uint32_t pos = base + mbcnt64(m);
            if (p[j] && pos < (uint32_t)kCandCap) {
                S.ckey[pos] = cand_key(__float_as_uint(e[j]), (uint32_t)(c0 + j));
                S.cval[pos] = __float_as_uint(e[j]);
            }
            base += (uint32_t)__builtin_popcountll(m);
        }
    }
}

// ---------------------------------------------------------------------------
// Per-group outlier choice (the outlier paragraph's own scope: the mask of
// every fixed quantization group keeps its k_g largest magnitudes, and the
// packet carries in-group offsets and fp16 values).  A group of g_q <= 256
// channels is 2^lv lanes of one wavefront, so the choice is wave-local.

// Signed max over the 2^lv lanes of an aligned block.
template <int LV>
__device__ __forceinline__ int32_t imax_lanes(int32_t v, int lv) {
    const int L = LV >= 0 ? LV : lv;
    auto dmax = [](int32_t a, int32_t b) { return a > b ? a : b; };
    if (L > 0) v = dmax(v, __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false));
    if (L > 1) v = dmax(v, __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false));
    if (L > 2) v = dmax(v, __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false));
    if (L > 3) v = dmax(v, __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false));
    if (L > 4) {
        auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        v = dmax((int32_t)p[0], (int32_t)p[1]);
    }
    return v;
}

// One bit at the first lane of every aligned block of 2^lv lanes.
__device__ __forceinline__ uint64_t block_starts(int lv) {
    switch (lv) {
        case 0: return ~0ull;
        case 1: return 0x5555555555555555ull;
        case 2: return 0x1111111111111111ull;
        case 3: return 0x0101010101010101ull;
        case 4: return 0x0001000100010001ull;
        default: return 0x0000000100000001ull;
    }
}

// The lowest set bit of every aligned block of 2^lv bits of a lane mask.
// Each block less one, without a borrow crossing into the next block (the
// blocks' top bits are set before the subtraction and put right after it),
// clears the block's lowest set bit and sets the bits below it, so x & ~(x - 1)
// per block is that bit; a zero block gives zero.  Six scalar instructions.
__device__ __forceinline__ uint64_t block_firsts(uint64_t x, int lv, uint64_t starts) {
    if (lv == 0) return x;
    const uint64_t tops = starts << ((1 << lv) - 1);
    const uint64_t less = ((x | tops) - starts) ^ (tops & ~x);
    return x & ~less;
}

// Chooses the k_g outliers of the lane's group and returns the lane's mask of
// chosen channels (bit j = channel c0 + j).  k_g rounds, each taking the
// group's largest remaining |E| and, among the channels holding it, the
// lowest.  Magnitudes are compared as the integer patterns of |E|, a chosen
// channel drops to -1, so a zero residual still outranks it, and k_g < g_q
// leaves every round a candidate.  The lanes holding the group maximum are
// those whose own maximum equals it; the lowest of them in each group keeps
// its lowest channel holding it, a scalar walk over the wave-wide masks of
// the lanes whose channel j does.  The entries, (fp16 value | in-group offset
// << 16), go to `st` at their position in the chunk's part of the row: group
// by group, ascending offset inside a group.
template <int LV>
__device__ __forceinline__ uint32_t select_group_outliers(const float* e, int lv, int kg, uint32_t lane,
                                                          uint32_t* st) {
    const int L = LV >= 0 ? LV : lv;
    int32_t a[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) a[j] = (int32_t)(__float_as_uint(e[j]) & 0x7FFFFFFFu);
    const uint64_t starts = block_starts(L);
    for (int i = 0; i < kg; ++i) {
        int32_t lb = a[0];
#pragma unroll
        for (int j = 1; j < 8; ++j) lb = lb > a[j] ? lb : a[j];
        const int32_t m = imax_lanes<LV>(lb, L);
        uint64_t lanes = block_firsts(ballot(lb == m), L, starts);  // one lane per group
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint64_t hit = ballot(a[j] == m);
            a[j] = __builtin_amdgcn_inverse_ballot_w64(hit & lanes) ? -1 : a[j];
            lanes &= ~hit;
        }
    }
    uint64_t sel[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) sel[j] = ballot(a[j] == -1);
    uint32_t selm = 0u;
#pragma unroll
    for (int j = 0; j < 8; ++j) selm |= __builtin_amdgcn_inverse_ballot_w64(sel[j]) ? (1u << j) : 0u;
    // slot of the lane's first entry: chosen channels of the group's lower
    // lanes, summed bit by bit over ballots of the per-lane counts (k_g = 1:
    // the group's one entry)
    uint32_t slot = (lane >> L) * (uint32_t)kg;
    if (kg > 1) {
        const uint32_t cnt = (uint32_t)__builtin_popcount(selm);
        const uint32_t g0 = lane & ~((1u << L) - 1u);
        const uint64_t below = ((1ull << lane) - 1ull) & ~((1ull << g0) - 1ull);
        const int nb = kg >= 8 ? 4 : (kg >= 4 ? 3 : 2);
        for (int b = 0; b < nb; ++b)
            slot += (uint32_t)__builtin_popcountll(ballot((cnt >> b) & 1u) & below) << b;
    }
    const uint32_t o0 = (lane & ((1u << L) - 1u)) * 8u;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        if (sel[j] != 0ull && __builtin_amdgcn_inverse_ballot_w64(sel[j]))
            st[slot] = f16_rne(e[j]) | ((o0 + (uint32_t)j) << 16);
        slot += (selm >> j) & 1u;
    }
    return selm;
}

// Store the chunk's staged per-group entries (at most 128: k_g <= g_q / 4):
// lane l writes entries l and l + 64 of the chunk, fp16 values to `rv` and u8
// offsets to `ro` (the row's two arrays); `first` is the chunk's first entry
// in the row and `n` its entry count.  Four stores per lane whatever n is.
__device__ __forceinline__ void store_group_outliers(Rsrc rv, Rsrc ro, uint32_t first, uint32_t n, uint32_t lane,
                                                     const uint32_t* st) {
    const uint32_t v0 = st[lane], v1 = st[lane + kWave];
    wave_lds_sync();  // the slice is reused for the reconstruction
    const bool in0 = lane < n, in1 = lane + kWave < n;
    bstore16(rv, in0 ? (first + lane) * 2u : kOut, v0);
    bstore16(rv, in1 ? (first + lane + kWave) * 2u : kOut, v1);
    bstore8(ro, in0 ? first + lane : kOut, v0 >> 16);
    bstore8(ro, in1 ? first + lane + kWave : kOut, v1 >> 16);
}

// ---------------------------------------------------------------------------
// Per-token outlier choice: the k largest |E| of the row, ties to the lower
// channel.  Called by every wavefront of the workgroup with its 8 residuals
// per lane; returns the per-lane mask of chosen channels (bit j = channel
// c0 + j) and writes the row's outlier entries in ascending channel order.
//
// 1. Threshold L: the channels of lane l in all wavefronts form one strided
//    group (64 channels spread over the row); its max |E| is built with one
//    LDS atomic max per lane.  Every wave finds the k-th largest of the 64
//    group maxima by an MSB-first radix select on the bit patterns (compare +
//    ballot per bit), stopping after the top 16 bits, which can only lower L.
//    At least k groups have a maximum >= L, each holding an element >= L, so
//    every outlier satisfies |E| >= L.  On the benchmark data about k+1
//    elements pass.
// 2. Candidates |E| >= L are appended to LDS.
// 3a. At most 64 candidates: wave 0 ranks their keys (|E|, -channel); rank
//     k-1 is the threshold key K*, outliers are the keys >= K*.
// 3b. Otherwise (heavy ties) the threshold is found directly: a radix select
//     of T = k-th largest |E| with workgroup-wide counts, then the last tied
//     channel c* by bisection on the channel among the elements equal to T.
// 4. An element is an outlier iff |E| > T, or |E| == T and channel <= c*.

__device__ __forceinline__ uint32_t select_outliers(const Args& A, RowShared& S, RowShared& Snext,
                                                    const float* e, bool act, int c0, uint32_t lane, int w,
                                                    uint32_t row) {
    const int k = A.k;
    // 1. strided group maxima: lane l of every wave -> one LDS max per lane
    float lm = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) lm = __builtin_fmaxf(lm, __builtin_fabsf(e[j]));
    if (act) atomicMax(&S.smax[lane], __float_as_uint(lm));  // bits order like non-negative floats
    __syncthreads();
    // The other buffer was last used by the previous row, which every wave
    // has finished: clear it for the next row.
    if (w == 0) {
        Snext.smax[lane] = 0u;
        if (lane < 4u) Snext.cnt[lane] = 0u;
    }
    // k-th largest of the 64 group maxima, top 16 bits (every wave, same result)
    const uint32_t v = S.smax[lane];
    uint32_t L = 0u;
#pragma unroll
    for (int bit = 30; bit >= 15; --bit) {
        const uint32_t c = L | (1u << bit);
        if ((uint32_t)__builtin_popcountll(ballot(v >= c)) >= (uint32_t)k) L = c;
    }
    const float Lf = __uint_as_float(L);
    // 2. candidates |E| >= L
    {
        bool p[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) p[j] = act & (__builtin_fabsf(e[j]) >= Lf);
        append8(S, &S.cnt[0], e, p, c0, lane);
    }
    __syncthreads();
    const uint32_t C = S.cnt[0];
    const Rsrc outl = rsrc(A.outl, (uint64_t)row * (uint64_t)k, (uint32_t)k * 4u);
    uint32_t T, cstar;
    bool ties;
    if (C <= (uint32_t)kCandCap) {
        // 3a. every wave ranks the candidates (one per lane) and finds K*
        // (rank = number of larger keys; keys are distinct as they hold the
        // channel; LDS broadcast reads, two keys at a time)
        const bool have = lane < C;
        const uint64_t key = have ? S.ckey[lane] : 0ull;
        uint32_t rank = 0;
        for (uint32_t j = 0; j < C; j += 2) {
            const ulonglong2 kk = *reinterpret_cast<const ulonglong2*>(&S.ckey[j]);
            rank += (kk.x > key) ? 1u : 0u;
            rank += (j + 1u < C && kk.y > key) ? 1u : 0u;
        }
        const uint64_t at = ballot(have && rank == (uint32_t)(k - 1));
        const uint64_t kst = rdlane64(key, at ? (int)__builtin_ctzll(at) : 0);
        T = (uint32_t)(kst >> 32);
        cstar = key_channel(kst);
        ties = __builtin_popcountll(ballot(have && (uint32_t)(key >> 32) >= T)) > (unsigned)k;
        if (w == 0) {
            // wave 0 writes the row's outliers in ascending channel order
            // (slot = number of chosen keys of a lower channel, i.e. of a
            // larger low word)
            const uint32_t ch = key_channel(key);
            uint32_t slot = 0;
            for (uint32_t j = 0; j < C; j += 2) {
                const ulonglong2 kk = *reinterpret_cast<const ulonglong2*>(&S.ckey[j]);
                slot += (kk.x >= kst && (uint32_t)kk.x > (uint32_t)key) ? 1u : 0u;
                slot += (j + 1u < C && kk.y >= kst && (uint32_t)kk.y > (uint32_t)key) ? 1u : 0u;
            }
            bstore32(outl, (have && key >= kst && slot < (uint32_t)k) ? slot * 4u : kOut,
                     ch | (f16_rne(__uint_as_float(S.cval[lane])) << 16));
        }
    } else {
        // 3b. radix select of T with workgroup-wide counts
        int it = 0;
        T = 0u;
        for (int bit = 30; bit >= 0; --bit) {
            const uint32_t c = T | (1u << bit);
            if (block_sum(S, count8(e, act, __uint_as_float(c)), it) >= (uint32_t)k) T = c;
        }
        const float Tf = __uint_as_float(T);
        uint32_t gtw = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) gtw += (uint32_t)__builtin_popcountll(ballot(act & (__builtin_fabsf(e[j]) > Tf)));
        const uint32_t gt = block_sum(S, gtw, it);
        const uint32_t ge = block_sum(S, count8(e, act, Tf), it);
        ties = ge != (uint32_t)k;
        cstar = 0xFFFFu;
        if (ties) {
            // smallest channel c* with count(|E| == T, channel <= c*) == k - gt
            const uint32_t need = (uint32_t)k - gt;
            uint32_t lo = 0u, hi = (uint32_t)A.d - 1u;
            while (lo < hi) {
                const uint32_t mid = (lo + hi) >> 1;
                uint32_t n = 0;
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    n += (uint32_t)__builtin_popcountll(
                        ballot(act & (__builtin_fabsf(e[j]) == Tf) & ((uint32_t)(c0 + j) <= mid)));
                if (block_sum(S, n, it) >= need) hi = mid;
                else lo = mid + 1u;
            }
            cstar = lo;
        }
        // gather the k outliers; wave 0 writes them by ascending channel
        const uint32_t cmax = ties ? cstar : 0xFFFFu;
        const int slot = 1 + it % 3;
        if (threadIdx.x == 0) S.cnt[1 + (it + 1) % 3] = 0u;
        __syncthreads();
        bool p[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float a = __builtin_fabsf(e[j]);
            p[j] = act & ((a > Tf) | ((a == Tf) & ((uint32_t)(c0 + j) <= cmax)));
        }
        append8(S, &S.cnt[slot], e, p, c0, lane);
        __syncthreads();
        if (w == 0) {
            const bool have = lane < (uint32_t)k;
            const uint32_t ch = have ? key_channel(S.ckey[lane]) : 0u;
            const uint32_t val = have ? S.cval[lane] : 0u;
            uint32_t pos = 0;
            for (int j = 0; j < k; ++j) pos += (key_channel(S.ckey[j]) < ch) ? 1u : 0u;
            bstore32(outl, (have && pos < (uint32_t)k) ? pos * 4u : kOut,
                     ch | (f16_rne(__uint_as_float(val)) << 16));
        }
    }
    // 4. mark this lane's outliers: |E| > T, or |E| == T and channel <= c*
    // when the cut falls inside a tie (bitwise, not short-circuit, logic:
    // the branches of && and || cost more than the comparisons)
    const float Tf = __uint_as_float(T);
    const uint32_t cmax = ties ? cstar : 0xFFFFu;
    uint32_t selm = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float a = __builtin_fabsf(e[j]);
        const bool p = act & ((a > Tf) | ((a == Tf) & ((uint32_t)(c0 + j) <= cmax)));
        if (p) selm |= 1u << j;
    }
    return selm;
}

// ---------------------------------------------------------------------------
// Encode with fused sender reconstruction.  One workgroup per token row (rows
// beyond the grid are taken in strides, the next row's x and ref prefetched
// into registers while the current one is processed), one wavefront per
// 512-channel chunk.

// GA / GQ select the group shape at compile time: 0..6 = groups inside one
// chunk with that many butterfly levels, 7 = groups spanning chunks, -1 =
// read from the arguments at run time.  OM is the outlier mode: 0 none, 1 the
// k largest |E| per token row, 2 the k_g largest per quantization group.
template <int BITS, int GA, int GQ, int OM>
__global__ __launch_bounds__(kWave * kMaxWaves) __attribute__((amdgpu_waves_per_eu(OM == 2 && GQ >= 0 ? 6 : 1)))
void rac_encode_kernel(Args A) {
    // LDS state of a row, double-buffered by row parity: every row that uses
    // LDS has a workgroup barrier, so no wave is more than one row ahead.
    __shared__ RowShared SS[2];
    extern __shared__ float4 XT[];  // per-wavefront store staging, kSlice each (sized at launch)
    const uint32_t lane = threadIdx.x & (kWave - 1);
    const int w = (int)(threadIdx.x / kWave);
    const int d = A.d;
    const int c0 = w * kChunk + (int)lane * 8;
    const bool act = c0 < d;
    constexpr float q = (float)((1 << (BITS - 1)) - 1);
    constexpr float inv_q = 1.0f / q;
    const int32_t fix = first_ref_index(A);  // store row of the first row's reference
    if (A.write_header && blockIdx.x == 0 && w == 0) write_header(A, lane);
    const bool dword3 = (d & 31) == 0;
    const bool multi_a = GA == 7 || (GA < 0 && A.lg_cpg_a > 0);
    const bool multi_q = GQ == 7 || (GQ < 0 && A.lg_cpg_q > 0);
    const int lv_a = GA >= 0 ? (GA == 7 ? 6 : GA) : A.lane_lv_a;
    const int lv_q = GQ >= 0 ? (GQ == 7 ? 6 : GQ) : A.lane_lv_q;
    const int grp_a = c0 >> A.lg_a, grp_q = c0 >> A.lg_q;
    const int cpg_a = 1 << A.lg_cpg_a, cpg_q = 1 << A.lg_cpg_q;
    const bool first_a = !multi_a ? (lane & ((1u << lv_a) - 1u)) == 0u : (lane == 0u && (w & (cpg_a - 1)) == 0);
    const bool first_q = !multi_q ? (lane & ((1u << lv_q) - 1u)) == 0u : (lane == 0u && (w & (cpg_q - 1)) == 0);
    const uint32_t sh_fixed = (A.fixed && act) ? step_roundup(A.steps[grp_q]) : 0u;
    const uint32_t ngq = (uint32_t)d >> A.lg_q, nga = (uint32_t)d >> A.lg_a;
    // per-group outliers: entries per row, this chunk's first entry and count
    const uint32_t gent = (uint32_t)A.k * ngq;
    const uint32_t gfirst = ((uint32_t)(w * kChunk) >> A.lg_q) * (uint32_t)A.k;
    const uint32_t gcount = ((uint32_t)__builtin_elementwise_min(kChunk, d - w * kChunk) >> A.lg_q) * (uint32_t)A.k;

    if (OM == 1) {
        if (w == 0) {
            SS[0].smax[lane] = 0u;
            SS[1].smax[lane] = 0u;
            if (lane < 4u) {
                SS[0].cnt[lane] = 0u;
                SS[1].cnt[lane] = 0u;
            }
        }
        __syncthreads();
    }
    // x and ref of row `rw` for this lane (zeros past the last row, past the
    // end of the row and for a zero reference)
    const uint32_t row_bytes = (uint32_t)d * 2u;
    // (nn: the row's position among the workgroup's rows)
    auto load_row = [&](uint32_t rw, int32_t ix, uint4& vx, uint4& vr) {
        const bool in = rw < A.tokens;
        const uint64_t o = (uint64_t)(in ? rw : 0) * (uint64_t)d;
        vx = bload128(rsrc(A.x, o, in ? row_bytes : 0u), (uint32_t)c0 * 2u);
        vr = bload128(ref_row(A, rw, in, ix), (uint32_t)c0 * 2u);
    };
    uint32_t row = blockIdx.x;
    uint4 nx, nr;
    const int32_t rix = load_ref_rows_v(A, lane);  // store rows of the gathered reference
    load_row(row, fix, nx, nr);
    // Let the first row land before the loop: then the loop head holds no
    // wait, and inside the loop only the prefetched loads are waited for
    // (never the stores of the row before).
    __builtin_amdgcn_s_waitcnt(kWaitVmem0);
    for (uint32_t n = 0; row < A.tokens; row += gridDim.x, ++n) {
        RowShared& S = SS[n & 1];
        const uint4 xv = nx, rv = nr;
        load_row(row + gridDim.x, ref_index_v(A, rix, n + 1u), nx, nr);
        float r[8], x[8];
        widen8(rv, r);
        widen8(xv, x);

        // a2: grouped affine fit, two-pass centred moments, pairwise sums
        float mr, mx, crr, crx;
        float uu[8], uv[8];
        if (!multi_a) {
            constexpr int L = GA == 7 ? 6 : GA;
            mr = lsum<L>(tree8(r), lv_a) * A.inv_ga;
            mx = lsum<L>(tree8(x), lv_a) * A.inv_ga;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float u = r[j] - mr, v = x[j] - mx;
                uu[j] = u * u;
                uv[j] = u * v;
            }
            crr = lsum<L>(tree8(uu), lv_a);
            crx = lsum<L>(tree8(uv), lv_a);
        } else {
            const int g0 = w & ~(cpg_a - 1);
            const float sr = lsum<6>(tree8(r), 6), sx = lsum<6>(tree8(x), 6);
            if (lane == 0u) {
                S.part[0][w] = sr;
                S.part[1][w] = sx;
            }
            __syncthreads();
            mr = tree_n(&S.part[0][g0], cpg_a) * A.inv_ga;
            mx = tree_n(&S.part[1][g0], cpg_a) * A.inv_ga;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float u = r[j] - mr, v = x[j] - mx;
                uu[j] = u * u;
                uv[j] = u * v;
            }
            const float suu = lsum<6>(tree8(uu), 6), suv = lsum<6>(tree8(uv), 6);
            if (lane == 0u) {
                S.part[2][w] = suu;
                S.part[3][w] = suv;
            }
            __syncthreads();
            crr = tree_n(&S.part[2][g0], cpg_a);
            crx = tree_n(&S.part[3][g0], cpg_a);
        }
        const uint32_t cf = A.cf_given ? bload32(rsrc(A.coef, (uint64_t)row * nga, nga * 4u), (uint32_t)grp_a * 4u)
                                       : fit_coef(crr, crx, mr, mx);
        bstore32(rsrc(A.coef, (uint64_t)row * nga, nga * 4u), (first_a && !A.cf_given) ? (uint32_t)grp_a * 4u : kOut, cf);

        // a3: aligned reference R~ = fma(alpha, r, beta) and residual E = x - R~
        const float a = f16_wire(cf & 0xFFFFu), b0 = f16_wire(cf >> 16);
        float rt[8], e[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            rt[j] = __builtin_fmaf(a, r[j], b0);
            e[j] = x[j] - rt[j];
        }

        // a4: outliers
        uint32_t selm = 0;
        if constexpr (OM == 1) selm = select_outliers(A, S, SS[(n + 1) & 1], e, act, c0, lane, w, row);
        if constexpr (OM == 2) {
            uint32_t* st = reinterpret_cast<uint32_t*>(XT + w * kSlice);
            selm = select_group_outliers<GQ>(e, lv_q, A.k, lane, st);
            wave_lds_sync();
            store_group_outliers(rsrc(A.gval, (uint64_t)row * gent, gent * 2u), rsrc(A.goff, (uint64_t)row * gent, gent),
                                 gfirst, gcount, lane, st);
        }
        float ed[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) ed[j] = e[j];
        if (selm) {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if ((selm >> j) & 1u) {
                    ed[j] = 0.0f;
                    // per-group mode: R~ of a chosen channel becomes its
                    // reconstruction R~ + O-hat now, so E is dead from here on
                    if constexpr (OM == 2) rt[j] = rt[j] + f16_wire(f16_rne(e[j]));
                }
        }

        // a5: scale of the quantization group
        uint32_t sh;
        if (A.fixed) {
            sh = sh_fixed;
        } else {
            float m = 0.0f;
#pragma unroll
            for (int j = 0; j < 8; ++j) m = __builtin_fmaxf(m, __builtin_fabsf(ed[j]));
            if (!multi_q) {
                m = lmax<GQ == 7 ? 6 : GQ>(m, lv_q);
            } else {
                m = lmax<6>(m, 6);
                if (lane == 0u) S.part[4][w] = m;
                __syncthreads();
                m = max_n(&S.part[4][w & ~(cpg_q - 1)], cpg_q);
            }
            sh = m == 0.0f ? 0u : scale_roundup(m, q, inv_q);
            bstore16(rsrc(A.scale, (uint64_t)row * ngq, ngq * 2u), first_q ? (uint32_t)grp_q * 2u : kOut, sh);
        }
        const float s = f16_wire(sh);
        const float inv = sh ? __builtin_amdgcn_rcpf(s) : 0.0f;

        // a6-a8: quantize (round half to even), pack, reconstruct
        float tc[8], mg[8], qf[8];
        float dist = 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            tc[j] = __builtin_amdgcn_fmed3f(ed[j] * inv, -q, q);
            mg[j] = tc[j] + kMagic;
            qf[j] = mg[j] - kMagic;
            dist = __builtin_fmaxf(dist, __builtin_fabsf(tc[j] - qf[j]));
        }
        if (dist > kNearHalf) {  // some quotient is near a tie: use the exact one
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (__builtin_fabsf(tc[j] - qf[j]) > kNearHalf) {
                    tc[j] = __builtin_amdgcn_fmed3f(ed[j] / s, -q, q);
                    mg[j] = tc[j] + kMagic;
                    qf[j] = mg[j] - kMagic;
                }
        }
        Packed<BITS> pk{};
        float H[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            pack_put<BITS>(pk, j, __float_as_uint(mg[j]));
            H[j] = __builtin_fmaf(qf[j], s, rt[j]);  // q*s is exact, so this is R~ + q*s
        }
        if (selm) {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if ((selm >> j) & 1u) H[j] = OM == 2 ? rt[j] : rt[j] + f16_wire(f16_rne(e[j]));
        }
        const uint32_t crb = (uint32_t)A.code_row_bytes;
        store_codes<BITS>(rsrc(A.codes, (uint64_t)row * crb, crb), w, lane, dword3, pk);
        store_xhat_t(xhat_row(A, row), A.xhat_bf16 != 0, (uint32_t)(w * kChunk), lane, XT + w * kSlice, H);
    }
}

// ---------------------------------------------------------------------------
// Encode with per-token outliers, NW wavefronts per token row.  For rows of
// at most NW * CPW * 512 channels whose groups lie inside a chunk, a
// workgroup of NW wavefronts owns one token row at a time and wavefront w
// holds the CPW chunks w, w + NW, ...: lane l keeps ref (as loaded) and the
// coefficient pair of channels [512c + 8l, 512c + 8l + 8) of its chunks in
// registers and their E in LDS, where the chunk's reconstruction is later
// staged for the store.  Keeping E out of registers leaves room to prefetch
// the next row (x once the fit is done, each ref chunk once its R~ is
// formed) at seven (CPW = 2) or five (CPW = 4) wavefronts per SIMD.  The
// per-token outlier choice costs
// two barriers between NW wavefronts, and its threshold search and ranking
// run NW times per row instead of once per chunk.

constexpr int kRowsWaves = 4;               // wavefronts per row
constexpr int kRowsMaxD = 16 * kChunk;       // channels per row (4 chunks per wavefront)
constexpr int kKeyChBits = 13;               // channel bits of the exact search's key (d <= 8192)
constexpr int kTop1 = 16;  // largest k whose first threshold comes from one maximum per lane
constexpr int kTop2 = 48;  // largest k whose first threshold takes two per wavefront lane (beyond: four)

// The third and fourth largest |E| of each (wavefront, lane), kept only with
// the larger candidate list.
template <int NW, bool MORE>
struct LaneMaxMore {
    uint32_t smax3[NW][kWave];
    uint32_t smax4[NW][kWave];
};
template <int NW>
struct LaneMaxMore<NW, false> {};

template <int NW, int CAP = kCandCap>
struct alignas(16) GroupShared : LaneMaxMore<NW, (CAP > kCandCap)> {
    static constexpr int cap = CAP;  // candidate list capacity
    // (ckey and cval, contiguous, also hold the exact search's three
    // 64-bin histograms while the list is dropped)
    uint64_t ckey[CAP];  // candidates: |E| bits << 32 | (0xFFFF - channel)
    uint32_t cval[CAP];  // their E bits
    uint32_t crw[CAP];   // their ref word (the bf16 pair holding the channel)
    uint32_t ccf[CAP];   // their group's coefficient pair
    uint32_t smax[NW][kWave]; // lane maxima of |E| of each wavefront
    uint32_t smax2[NW][kWave];// the lanes' second largest |E| (k > kTop1)
    uint32_t thr;             // that threshold, from wavefront 0
    uint32_t cnt[2];          // candidate count (LDS atomic), by row parity
    uint32_t xn[2];           // count of the rebuilt list (exact search), by row parity
};
static_assert(offsetof(GroupShared<4>, cval) == sizeof(uint64_t) * kCandCap &&
                  sizeof(uint64_t) * kCandCap + sizeof(uint32_t) * kCandCap >= 3 * kWave * sizeof(uint32_t),
              "the histograms of the exact search fit in ckey and cval");

// Append this lane's elements of one chunk whose |E| pattern is >= lo (and,
// with use_key, whose key is >= kmin) to the shared candidate list, with
// what R~ is formed from (the loaded ref word and the coefficient pair
// cfv); one LDS atomic per wavefront reserves the slots, entries beyond the
// list's capacity are counted but not stored.
template <class G>
__device__ __forceinline__ void append_shared(G& S, uint32_t* counter,
                                              const float* e, const uint4& rpk, uint32_t cfv, bool act, uint32_t c0,
                                              uint32_t lo, bool use_key, uint64_t kmin, uint32_t lane) {
    bool p[8];
    uint32_t n = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint32_t eb = __float_as_uint(e[j]);
        p[j] = act & ((eb & 0x7FFFFFFFu) >= lo) & (!use_key | (cand_key(eb, c0 + j) >= kmin));
        n += (uint32_t)__builtin_popcountll(ballot(p[j]));
    }
    if (!n) return;
    uint32_t base = 0u;
    if (lane == 0u) base = atomicAdd(counter, n);
    base = uniform(base);
    const uint32_t rw[4] = {rpk.x, rpk.y, rpk.z, rpk.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint64_t m = ballot(p[j]);
        if (m) {
            const uint32_t pos = base + mbcnt64(m);
            if (p[j] & (pos < (uint32_t)G::cap)) {
                S.ckey[pos] = cand_key(__float_as_uint(e[j]), c0 + j);
                S.cval[pos] = __float_as_uint(e[j]);
                S.crw[pos] = rw[j >> 1];
                S.ccf[pos] = cfv;
            }
            base += (uint32_t)__builtin_popcountll(m);
        }
    }
}

// The same for the candidate rule |E| >= Lf alone (the threshold search's
// bound), with float compares on |E| (inputs are finite, so E is never NaN and
// the float order of |E| is the order of its bit patterns).  A lane's mask
// bit comes from its compare ANDed with the wavefront's active-lane mask
// (ballot of act), so each element costs one vector compare.
template <class G>
__device__ __forceinline__ void append_bound(G& S, uint32_t* counter, const float* e, const uint4& rpk, uint32_t cfv,
                                             bool act, uint32_t c0, float Lf, uint32_t lane) {
    const uint64_t actm = ballot(act);
    uint32_t n = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) n += (uint32_t)__builtin_popcountll(ballot(__builtin_fabsf(e[j]) >= Lf) & actm);
    if (!n) return;
    uint32_t base = 0u;
    if (lane == 0u) base = atomicAdd(counter, n);
    base = uniform(base);
    const uint32_t rw[4] = {rpk.x, rpk.y, rpk.z, rpk.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint64_t m = ballot(__builtin_fabsf(e[j]) >= Lf) & actm;
        if (m) {
            const uint32_t pos = base + mbcnt64(m);
            if (act & (__builtin_fabsf(e[j]) >= Lf) & (pos < (uint32_t)G::cap)) {
                S.ckey[pos] = cand_key(__float_as_uint(e[j]), c0 + j);
                S.cval[pos] = __float_as_uint(e[j]);
                S.crw[pos] = rw[j >> 1];
                S.ccf[pos] = cfv;
            }
            base += (uint32_t)__builtin_popcountll(m);
        }
    }
}

// Pooled fit: the first row of the segment holding token row `row`, that is
// seg_start[s] for the largest s < segments with seg_start[s] <= row.  The
// search takes 64 starts per level (one vector load, then the highest lane of
// a ballot: the sorted starts at or below the row are a prefix of the
// lanes), so up to 64 segments take one level and 4096 two.  The result is
// clamped to [0, tokens - 1]: whatever the starts hold, the row read stays in
// the coefficient section.
__device__ __forceinline__ uint32_t seg_first_row(const Args& A, uint32_t row) {
    const uint32_t lane = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
    int64_t base = 0, span = A.segments;
    int32_t f = 0;
    for (;;) {
        const int64_t stride = (span + kWave - 1) / kWave;
        const int64_t idx = base + (int64_t)lane * stride;
        const int32_t v = idx < base + span ? A.seg_start[idx] : INT32_MAX;
        const uint64_t le = ballot(v <= (int32_t)row);
        const int c = le ? 63 - __builtin_clzll(le) : 0;
        base += (int64_t)c * stride;
        if (stride == 1) {
            f = (int32_t)rdlane((uint32_t)v, c);
            break;
        }
        span = stride < A.segments - base ? stride : A.segments - base;
    }
    f = f < 0 ? 0 : f;
    return (uint32_t)f < A.tokens ? (uint32_t)f : A.tokens - 1u;
}

// Hide held ref values from the optimizer before they are widened again (a
// reused widening would keep 8 more registers per chunk alive across the row).
template <int N>
__device__ __forceinline__ void opaque_n(uint4 (&r)[N]) {
#pragma unroll
    for (int i = 0; i < N; ++i) asm volatile("" : "+v"(r[i].x), "+v"(r[i].y), "+v"(r[i].z), "+v"(r[i].w));
}

// GIVEN: the wire already holds every row's (alpha, beta) (pooled fit), which
// is read instead of fitted.
// TWO: the first outlier threshold from the two largest |E| of each
// (wavefront, lane) (for kTop1 < k <= kTop2; a separate kernel, so that the
// other k keep the code and registers of the one-value bound).
// BIG: the first threshold from the four largest |E| of each (wavefront,
// lane) and a candidate list of 2 * kCandCap entries, ranked two per lane
// (for k > kTop2, whose rows would overflow the smaller list almost always).
template <int BITS, int GA, int GQ, int NW, int CPW, bool GIVEN, bool TWO, bool BIG = false>
__global__ __launch_bounds__(NW * kWave) __attribute__((amdgpu_waves_per_eu(CPW == 2 ? (BIG ? 6 : 7) : 4)))
void rac_encode_rows_kernel(Args A) {
    // (a row's lists are read before the next row's first barrier and
    // written after it; only the count is reset early, so it alternates)
    __shared__ GroupShared<NW, BIG ? 2 * kCandCap : kCandCap> S;
    // E of each wavefront's chunks (one slice per chunk), later the staging
    // of the chunk's reconstruction
    __shared__ float4 EL[NW][CPW][kSlice];
    const uint32_t lane = threadIdx.x & (kWave - 1);
    const int w = (int)uniform(threadIdx.x / kWave);
    const int d = A.d, k = A.k;
    constexpr float q = (float)((1 << (BITS - 1)) - 1);
    constexpr float inv_q = 1.0f / q;
    if (A.write_header && blockIdx.x == 0 && w == 0) write_header(A, lane);
    const bool dword3 = (d & 31) == 0;
    const int lv_a = GA >= 0 ? GA : A.lane_lv_a;
    const int lv_q = GQ >= 0 ? GQ : A.lane_lv_q;
    const uint32_t ngq = (uint32_t)d >> A.lg_q, nga = (uint32_t)d >> A.lg_a;
    const uint32_t row_bytes = (uint32_t)d * 2u;
    const uint32_t crb = (uint32_t)A.code_row_bytes;
    // first channel of the wavefront's i-th chunk: chunks are dealt round the
    // wavefronts, so a row of fewer than NW * CPW chunks stays balanced
    auto chunk_at = [&](int i) { return (w + i * NW) * kChunk; };
    const int32_t rix = load_ref_rows_v(A, lane);  // store rows of the gathered reference
    const int32_t fix = first_ref_index(A);
    if (w == 0 && lane < 2u) {
        S.cnt[lane] = 0u;
        S.xn[lane] = 0u;
    }
    __syncthreads();

    // x and ref of the block's first row; later rows are prefetched into
    // the same registers as they fall free (x after the fit, each ref chunk
    // after its R~ is formed), ahead of the current row's stores
    uint4 xl[CPW], rp[CPW];
    {
        const uint32_t row = blockIdx.x;
        const bool any = row < A.tokens;
        const uint64_t o = (uint64_t)row * (uint64_t)d;
        const Rsrc rx = rsrc(A.x, o, any ? row_bytes : 0u), rr = ref_row(A, row, any, fix);
#pragma unroll
        for (int i = 0; i < CPW; ++i) {
            const uint32_t off = ((uint32_t)(chunk_at(i)) + lane * 8u) * 2u;  // past the row: reads 0
            xl[i] = bload128(rx, off);
            rp[i] = bload128(rr, off);
        }
    }
    // A store that the range check drops, so that stores are outstanding at
    // the loop entry as they are at the end of every row: the compiler's wait
    // analysis then keeps the memory operations in order across the loop and
    // the fit waits for the prefetched loads, not for the previous row's
    // stores issued after them.
    bstore32(rsrc(A.coef, 0, 0u), kOut, 0u);

    uint32_t n = 0;
    for (uint32_t row = blockIdx.x; row < A.tokens; row += gridDim.x, ++n) {
        uint32_t* const cnt = &S.cnt[n & 1];
        // lane * 8, opaque inside the loop: otherwise every per-channel
        // constant of the lane's channels is hoisted out of the row loop
        // (the lane id is recomputed, not kept live across the loop)
        uint32_t l8;
        asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0\n\tv_lshlrev_b32 %0, 3, %0"
                     : "=v"(l8));
        const uint32_t lane = l8 >> 3;  // (likewise every lane offset below)
        const bool first_a = (lane & ((1u << lv_a) - 1u)) == 0u;
        const bool first_q = (lane & ((1u << lv_q) - 1u)) == 0u;
        int d = A.d;  // (per row as well: tests on it stay scalar instead of being kept in registers)
        asm volatile("" : "+s"(d));
        const uint32_t nrow = row + gridDim.x;
        const bool more = nrow < A.tokens;
        const uint64_t on = (uint64_t)nrow * (uint64_t)d;
        const Rsrc nx = rsrc(A.x, on, more ? row_bytes : 0u), nr = ref_row(A, nrow, more, ref_index_v(A, rix, n + 1u));
        uint32_t cf[CPW];
#pragma unroll
        for (int i = 0; i < CPW; ++i) cf[i] = 0u;

        // a2-a3 per chunk: fit of the lane's group, E; lane maxima of |E|
        // (per chunk, and over the wavefront's chunks)
        const Rsrc rcoef = rsrc(A.coef, (uint64_t)row * nga, nga * 4u);
        // pooled fit: the pair is read from the first row of the row's segment
        const uint32_t frow = GIVEN ? seg_first_row(A, row) : row;
        const Rsrc rgiven = rsrc(A.coef, (uint64_t)frow * nga, GIVEN ? nga * 4u : 0u);
        float lmc[CPW];
#pragma unroll
        for (int i = 0; i < CPW; ++i) lmc[i] = 0.0f;
#pragma unroll
        for (int i = 0; i < CPW; ++i) {
            if (chunk_at(i) >= d) continue;
            const uint32_t c0 = (uint32_t)(chunk_at(i)) + l8;
            float r[8], x[8], uu[8], uv[8];
            widen8(rp[i], r);
            widen8(xl[i], x);
            const float mr = lsum<GA>(tree8(r), lv_a) * A.inv_ga;
            const float mx = lsum<GA>(tree8(x), lv_a) * A.inv_ga;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float u = r[j] - mr, v = x[j] - mx;
                uu[j] = u * u;
                uv[j] = u * v;
            }
            const float crr = lsum<GA>(tree8(uu), lv_a), crx = lsum<GA>(tree8(uv), lv_a);
            if constexpr (GIVEN) {
                cf[i] = bload32(rgiven, (c0 >> A.lg_a) * 4u);
                bstore32(rcoef, first_a ? (c0 >> A.lg_a) * 4u : kOut, cf[i]);
            } else {
                cf[i] = fit_coef(crr, crx, mr, mx);
                bstore32(rcoef, first_a ? (c0 >> A.lg_a) * 4u : kOut, cf[i]);
            }
            const float a = f16_wire(cf[i] & 0xFFFFu), b0 = f16_wire(cf[i] >> 16);
            float e[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {  // E = 0 past the row
                e[j] = x[j] - __builtin_fmaf(a, r[j], b0);
                lmc[i] = __builtin_fmaxf(lmc[i], __builtin_fabsf(e[j]));
            }
            put8(EL[w][i], lane, e);
        }
        float lmx = lmc[0];
#pragma unroll
        for (int i = 1; i < CPW; ++i) lmx = __builtin_fmaxf(lmx, lmc[i]);

#pragma unroll
        for (int i = 0; i < CPW; ++i) xl[i] = bload128(nx, ((uint32_t)(chunk_at(i)) + l8) * 2u);

        // a4: the k largest |E| of the row (ties to the lower channel).
        // Threshold L: the k-th largest of the 64 maxima of |E| over lane l
        // of all wavefronts, cut to its top 16 bits (which can only lower
        // it); each of >= k such groups holds an element >= L, so every
        // outlier has |E| >= L.  For kTop1 < k <= kTop2 each of the 64 groups
        // gives its two largest |E| (two distinct elements; from the two
        // largest of each wavefront's 16 channels of the lane): L is the
        // k-th largest of those 128 values, again with >= k elements >= L,
        // and on rows whose large |E| crowd into some channels far fewer
        // elements pass it (fewer rows overflow the candidate list).  Beyond
        // kTop2 (BIG) each group gives its four largest, L is the k-th
        // largest of those 256 values, and the list holds 2 * kCandCap.
        S.smax[w][lane] = __float_as_uint(lmx);
        constexpr bool two = TWO || BIG;
        if constexpr (BIG) {
            // the four largest (a multiset: ties count separately), each
            // value entering at the top and the smaller one moving down
            uint32_t m1 = 0u, m2 = 0u, m3 = 0u, m4 = 0u;
#pragma unroll
            for (int i = 0; i < CPW; ++i) {
                if (chunk_at(i) >= d) continue;
                float e[8];
                get8(EL[w][i], lane, e);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    uint32_t t = __float_as_uint(e[j]) & 0x7FFFFFFFu, hi;
                    hi = __builtin_elementwise_max(m1, t); t = __builtin_elementwise_min(m1, t); m1 = hi;
                    hi = __builtin_elementwise_max(m2, t); t = __builtin_elementwise_min(m2, t); m2 = hi;
                    hi = __builtin_elementwise_max(m3, t); t = __builtin_elementwise_min(m3, t); m3 = hi;
                    m4 = __builtin_elementwise_max(m4, t);
                }
            }
            S.smax2[w][lane] = m2;
            S.smax3[w][lane] = m3;
            S.smax4[w][lane] = m4;
        } else if constexpr (two) {
            uint32_t m1 = 0u, m2 = 0u;
#pragma unroll
            for (int i = 0; i < CPW; ++i) {
                if (chunk_at(i) >= d) continue;
                float e[8];
                get8(EL[w][i], lane, e);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const uint32_t b = __float_as_uint(e[j]) & 0x7FFFFFFFu;
                    m2 = __builtin_elementwise_max(m2, __builtin_elementwise_min(m1, b));
                    m1 = __builtin_elementwise_max(m1, b);
                }
            }
            S.smax2[w][lane] = m2;
        }
        __syncthreads();
        // the other buffer was last read by the previous row, which every
        // wavefront has left: reset its candidate count for the next row
        if (w == 0 && lane == 0u) {
            S.cnt[(n + 1) & 1] = 0u;
            S.xn[(n + 1) & 1] = 0u;
        }
        uint32_t v = S.smax[0][lane];
#pragma unroll
        for (int ww = 1; ww < NW; ++ww) v = __builtin_elementwise_max(v, S.smax[ww][lane]);
        uint32_t L = 0u;
        if constexpr (!two) {
#pragma unroll
            for (int bit = 30; bit >= 15; --bit) {
                const uint32_t cnd = L | (1u << bit);
                if ((uint32_t)__builtin_popcountll(ballot(v >= cnd)) >= (uint32_t)k) L = cnd;
            }
        } else {
            // wavefront 0 alone searches (its ballot counts are scalar work,
            // and the compute unit's scalar unit is shared by all its
            // wavefronts), then hands L over through LDS
            if (w == 0) {
                // the two (with BIG four) largest of the lane's values from
                // every wavefront: distinct elements of the 64 channels of
                // lane l in all wavefronts
                uint32_t a1 = 0u, a2 = 0u, a3 = 0u, a4 = 0u;
                auto insert = [&](uint32_t t) {
                    uint32_t hi;
                    hi = __builtin_elementwise_max(a1, t); t = __builtin_elementwise_min(a1, t); a1 = hi;
                    if constexpr (BIG) {
                        hi = __builtin_elementwise_max(a2, t); t = __builtin_elementwise_min(a2, t); a2 = hi;
                        hi = __builtin_elementwise_max(a3, t); t = __builtin_elementwise_min(a3, t); a3 = hi;
                        a4 = __builtin_elementwise_max(a4, t);
                    } else {
                        a2 = __builtin_elementwise_max(a2, t);
                    }
                };
#pragma unroll
                for (int ww = 0; ww < NW; ++ww) {
                    insert(S.smax[ww][lane]);
                    insert(S.smax2[ww][lane]);
                    if constexpr (BIG) {
                        insert(S.smax3[ww][lane]);
                        insert(S.smax4[ww][lane]);
                    }
                }
#pragma unroll
                for (int bit = 30; bit >= 15; --bit) {
                    const uint32_t cnd = L | (1u << bit);
                    uint32_t c = (uint32_t)__builtin_popcountll(ballot(a1 >= cnd)) +
                                 (uint32_t)__builtin_popcountll(ballot(a2 >= cnd));
                    if constexpr (BIG)
                        c += (uint32_t)__builtin_popcountll(ballot(a3 >= cnd)) +
                             (uint32_t)__builtin_popcountll(ballot(a4 >= cnd));
                    if (c >= (uint32_t)k) L = cnd;
                }
                if (lane == 0u) S.thr = L;
            }
            __syncthreads();
            L = uniform(S.thr);
        }
        opaque_n(rp);
        const float Lf = __uint_as_float(L);
#pragma unroll
        for (int i = 0; i < CPW; ++i) {
            // (a chunk none of whose lane maxima reaches L holds no candidate)
            if ((chunk_at(i) >= d) || !ballot(lmc[i] >= Lf)) continue;
            const uint32_t c0 = (uint32_t)(chunk_at(i)) + l8;
            float e[8];
            get8(EL[w][i], lane, e);
            append_bound(S, cnt, e, rp[i], cf[i], c0 < (uint32_t)d, c0, Lf, lane);
        }
        __syncthreads();
        // k-th largest of the first Cn listed keys (Cn <= S.cap; lane i
        // ranks key i, and with BIG key i + 64 as well, by the number of
        // larger keys, which are distinct; LDS broadcast reads, two keys at a
        // time); `key` and `key2` get lane i's keys
        auto kth_key = [&](uint32_t Cn, uint64_t& key, uint64_t& key2) -> uint64_t {
            const bool have = lane < Cn, have2 = BIG && lane + (uint32_t)kWave < Cn;
            key = have ? S.ckey[lane] : 0ull;
            key2 = have2 ? S.ckey[lane + kWave] : 0ull;
            uint32_t rank = 0, rank2 = 0;
            for (uint32_t j = 0; j < Cn; j += 2) {
                const ulonglong2 kk = *reinterpret_cast<const ulonglong2*>(&S.ckey[j]);
                const bool y = j + 1u < Cn;
                rank += (kk.x > key) ? 1u : 0u;
                rank += (y && kk.y > key) ? 1u : 0u;
                if constexpr (BIG) {
                    rank2 += (kk.x > key2) ? 1u : 0u;
                    rank2 += (y && kk.y > key2) ? 1u : 0u;
                }
            }
            const uint64_t at = ballot(have && rank == (uint32_t)(k - 1));
            if constexpr (BIG) {
                if (!at) {
                    const uint64_t at2 = ballot(have2 && rank2 == (uint32_t)(k - 1));
                    return rdlane64(key2, at2 ? (int)__builtin_ctzll(at2) : 0);
                }
            }
            return rdlane64(key, at ? (int)__builtin_ctzll(at) : 0);
        };
        // (values read from LDS are the same in every lane: readfirstlane
        // makes that visible, so the branches on them stay scalar)
        uint32_t C = uniform(*cnt);
        uint64_t key = 0ull;
        uint64_t kst = 0ull;  // the outliers are the listed keys >= kst
        if (C > (uint32_t)S.cap) {
            // More candidates than the list holds: they are narrowed by a
            // radix search over a 49-bit key (|E| pattern, 8191 - channel,
            // 5 zero bits; a larger key ranks higher), from the top digit
            // not shared by every candidate (all lie in [L, row maximum]).
            // Each digit (6 bits, the last one narrower) is taken from a
            // 64-bin histogram of the candidates that share the digits found
            // so far: the bin holding the k-th largest.  Once the keys in
            // that bin or above number at most S.cap, the list is rebuilt
            // from them and ranked as usual; keys are distinct, so at worst
            // the last digit gets there.  The histograms (three, in turn,
            // each cleared two levels before it is filled, so one barrier
            // per level) use the list's storage.
            uint32_t* const H = reinterpret_cast<uint32_t*>(S.ckey);  // [3][64]: ckey and cval
            if (threadIdx.x < 2u * kWave) H[threadIdx.x] = 0u;
            uint32_t mx = v;  // row maximum of the |E| patterns
#pragma unroll
            for (int o = 1; o < kWave; o <<= 1) mx = __builtin_elementwise_max(mx, (uint32_t)__shfl_xor((int)mx, o));
            mx = uniform(mx);
            const int hb = (mx == L) ? -1 : 31 - __builtin_clz(mx ^ L);  // highest bit not shared
            uint64_t prefix = (uint64_t)(L >> (hb + 1));
            constexpr uint32_t kChMax = (1u << kKeyChBits) - 1u;
            int shift = hb + kKeyChBits, width = 6;  // the digit just below the shared bits
            uint32_t need = (uint32_t)k;
            __syncthreads();
#pragma unroll 1
            for (int lev = 0;; ++lev) {
                uint32_t* const h = H + (lev % 3) * kWave;
                if (w == 0) H[((lev + 1) % 3) * kWave + lane] = 0u;
                // (one element at a time, read from the slices: this rare path
                // then needs few registers)
#pragma unroll 1
                for (int i = 0; i < CPW; ++i) {
                    const uint32_t c0 = (uint32_t)(chunk_at(i)) + l8;
                    if (c0 >= (uint32_t)d) continue;
                    const float* const es = reinterpret_cast<const float*>(EL[w][i]);
#pragma unroll 1
                    for (uint32_t j = 0; j < 8u; ++j) {
                        const uint32_t pa = __float_as_uint(es[slice_float(l8 + j)]) & 0x7FFFFFFFu;
                        const uint64_t key = ((uint64_t)pa << (kKeyChBits + 5)) | ((uint64_t)(kChMax - (c0 + j)) << 5);
                        if ((pa >= L) & ((key >> (shift + width)) == prefix))
                            atomicAdd(&h[(uint32_t)(key >> shift) & ((1u << width) - 1u)], 1u);
                    }
                }
                __syncthreads();
                // lane l takes bin 63 - l; inclusive sums from the top bin
                const uint32_t hv = h[kWave - 1 - lane];
                uint32_t P = hv;
#pragma unroll
                for (int o = 1; o < kWave; o <<= 1) {
                    const uint32_t t = (uint32_t)__shfl_up((int)P, o);
                    if (lane >= (uint32_t)o) P += t;
                }
                const int ls = (int)__builtin_ctzll(ballot(P >= need));  // some lane: the prefix holds >= need
                const uint32_t above = rdlane(P - hv, ls), nb = rdlane(hv, ls);
                prefix = (prefix << width) | (uint64_t)(kWave - 1 - ls);
                need -= above;
                // keys in this bin or above: k - need + nb
                if ((uint32_t)k - need + nb <= (uint32_t)S.cap || shift == 0) break;
                width = shift >= 6 ? 6 : shift;
                shift -= width;
            }
            // rebuild the list from the keys >= the bin's lowest: |E|
            // pattern > pm, or == pm and channel <= kChMax - cm
            const uint64_t kl = (prefix << shift) >> 5;
            const uint32_t pm = (uint32_t)(kl >> kKeyChBits), cm = (uint32_t)(kl & kChMax);
            const uint64_t kmin = ((uint64_t)pm << 32) | (uint64_t)(0xFFFFu - kChMax + cm);
            uint32_t* const xc = &S.xn[n & 1];
            __syncthreads();  // (every wavefront has read the last histogram)
#pragma unroll
            for (int i = 0; i < CPW; ++i) {
                const uint32_t c0 = (uint32_t)(chunk_at(i)) + l8;
                float e[8];
                get8(EL[w][i], lane, e);
                append_shared(S, xc, e, rp[i], cf[i], c0 < (uint32_t)d, c0, pm, true, kmin, lane);
            }
            __syncthreads();
            C = uniform(*xc);  // k <= C <= S.cap
        }
        uint64_t key2 = 0ull;
        kst = kth_key(C, key, key2);
        const bool have = lane < C;
        // Candidate lane i holds one chosen outlier (or none; with BIG two,
        // entries i and i + 64): its channel and its reconstruction
        // R~ + fp16(E), which phase C writes over the staged value of that
        // channel.  Every outlier is a candidate and keys are distinct, so
        // the outliers are exactly the candidate keys >= kst.
        const bool chosen = have && key >= kst;
        const uint32_t och = chosen ? key_channel(key) : 0xFFFFFFFFu;
        uint32_t oval = 0u;
        float ohat = 0.0f;
        if (chosen) {
            oval = f16_rne(__uint_as_float(S.cval[lane]));
            const uint32_t rw = S.crw[lane], cfc = S.ccf[lane];
            const float r = (och & 1u) ? bf16_hi(rw) : bf16_lo(rw);
            ohat = __builtin_fmaf(f16_wire(cfc & 0xFFFFu), r, f16_wire(cfc >> 16)) + f16_wire(oval);
        }
        bool chosen2 = false;
        uint32_t och2 = 0xFFFFFFFFu, oval2 = 0u;
        float ohat2 = 0.0f;
        if constexpr (BIG) {
            chosen2 = lane + (uint32_t)kWave < C && key2 >= kst;
            if (chosen2) {
                const uint32_t i2 = lane + (uint32_t)kWave;
                och2 = key_channel(key2);
                oval2 = f16_rne(__uint_as_float(S.cval[i2]));
                const uint32_t rw = S.crw[i2], cfc = S.ccf[i2];
                const float r = (och2 & 1u) ? bf16_hi(rw) : bf16_lo(rw);
                ohat2 = __builtin_fmaf(f16_wire(cfc & 0xFFFFu), r, f16_wire(cfc >> 16)) + f16_wire(oval2);
            }
        }
        if (w == 0) {
            // the row's outliers in ascending channel order (slot = number of
            // chosen keys of a lower channel, i.e. of a larger low word)
            uint32_t slot = 0, slot2 = 0;
            for (uint32_t j = 0; j < C; j += 2) {
                const ulonglong2 kk = *reinterpret_cast<const ulonglong2*>(&S.ckey[j]);
                const bool cx = kk.x >= kst, cy = j + 1u < C && kk.y >= kst;
                slot += (cx && (uint32_t)kk.x > (uint32_t)key) ? 1u : 0u;
                slot += (cy && (uint32_t)kk.y > (uint32_t)key) ? 1u : 0u;
                if constexpr (BIG) {
                    slot2 += (cx && (uint32_t)kk.x > (uint32_t)key2) ? 1u : 0u;
                    slot2 += (cy && (uint32_t)kk.y > (uint32_t)key2) ? 1u : 0u;
                }
            }
            const Rsrc outl = rsrc(A.outl, (uint64_t)row * (uint64_t)k, (uint32_t)k * 4u);
            bstore32(outl, (chosen && slot < (uint32_t)k) ? slot * 4u : kOut, key_channel(key) | (oval << 16));
            if constexpr (BIG)
                bstore32(outl, (chosen2 && slot2 < (uint32_t)k) ? slot2 * 4u : kOut, key_channel(key2) | (oval2 << 16));
        }

        // E^d: E with the outliers set to 0, in place (each wavefront
        // clears the outliers of its own chunks, which only it reads)
#pragma unroll
        for (int i = 0; i < CPW; ++i) {
            const uint32_t oc = och - (uint32_t)(chunk_at(i));
            if (oc < (uint32_t)kChunk) reinterpret_cast<float*>(EL[w][i])[slice_float(oc)] = 0.0f;
            if constexpr (BIG) {
                const uint32_t oc2 = och2 - (uint32_t)(chunk_at(i));
                if (oc2 < (uint32_t)kChunk) reinterpret_cast<float*>(EL[w][i])[slice_float(oc2)] = 0.0f;
            }
        }
        wave_lds_sync();

        // a5-a8 per chunk: scale, quantize, pack, reconstruct
        opaque_n(rp);
        const Rsrc rsc = rsrc(A.scale, (uint64_t)row * ngq, ngq * 2u);
        const Rsrc rcd = rsrc(A.codes, (uint64_t)row * crb, crb);
        const Rsrc rxh = xhat_row(A, row);
#pragma unroll
        for (int i = 0; i < CPW; ++i) {
            if (chunk_at(i) >= d) continue;
            const uint32_t chunk0 = (uint32_t)(chunk_at(i));
            const uint32_t c0 = chunk0 + l8;
            float ed[8];
            float4* st = EL[w][i];
            get8(st, lane, ed);  // (past the row E is 0)
            float m = 0.0f;
#pragma unroll
            for (int j = 0; j < 8; ++j) m = __builtin_fmaxf(m, __builtin_fabsf(ed[j]));
            m = lmax<GQ>(m, lv_q);
            const uint32_t sh = m == 0.0f ? 0u : scale_roundup(m, q, inv_q);
            bstore16(rsc, first_q ? (c0 >> A.lg_q) * 2u : kOut, sh);
            const float s = f16_wire(sh);
            const float inv = sh ? __builtin_amdgcn_rcpf(s) : 0.0f;
            // |E^d| <= s q, so E^d * (1/s) stays below q + 1/2 unless the
            // scale saturated; that case and quotients near a tie take the
            // clamped, correctly rounded path
            float mg[8], qf[8];
            float dist = 0.0f;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float t = ed[j] * inv;
                mg[j] = t + kMagic;
                qf[j] = mg[j] - kMagic;
                dist = __builtin_fmaxf(dist, __builtin_fabsf(t - qf[j]));
            }
            if ((dist > kNearHalf) | (sh == 0x7C00u)) {
                float inv2 = inv;
                asm volatile("" : "+v"(inv2));  // recomputed here rather than kept live
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const float t0 = ed[j] * inv2;
                    const float t = __builtin_fabsf(t0 - qf[j]) > kNearHalf ? ed[j] / s : t0;
                    mg[j] = __builtin_amdgcn_fmed3f(t, -q, q) + kMagic;
                    qf[j] = mg[j] - kMagic;
                }
            }
            float H[8];
            {
                float r[8];
                widen8(rp[i], r);
                const float a = f16_wire(cf[i] & 0xFFFFu), b0 = f16_wire(cf[i] >> 16);
#pragma unroll
                for (int j = 0; j < 8; ++j) H[j] = __builtin_fmaf(qf[j], s, __builtin_fmaf(a, r[j], b0));  // R~ + q*s (q*s exact)
            }
            rp[i] = bload128(nr, c0 * 2u);
            store_codes<BITS>(rcd, w + i * NW, lane, dword3, pack8<BITS>(mg));
            put8(st, lane, H);
            wave_lds_sync();
            if (och - chunk0 < (uint32_t)kChunk) reinterpret_cast<float*>(st)[slice_float(och - chunk0)] = ohat;
            if constexpr (BIG)
                if (och2 - chunk0 < (uint32_t)kChunk) reinterpret_cast<float*>(st)[slice_float(och2 - chunk0)] = ohat2;
            wave_lds_sync();
            emit_xhat(rxh, A.xhat_bf16 != 0, chunk0, l8 >> 3, st);
        }
    }
}

// ---------------------------------------------------------------------------
// Decode / reconstruct: one workgroup per token row (strided, with the next
// row's inputs prefetched), one wavefront per chunk, no cross-wave work.
// OM: the wire's outlier mode (0 none, 1 per token row, 2 per quantization
// group); BF16: the reconstruction is stored as bf16.  (Both are compile-time,
// so no branch separates a row's memory operations.)

template <int BITS, int OM, bool BF16>
__global__ __launch_bounds__(kWave * kMaxWaves) void rac_decode_kernel(Args A) {
    extern __shared__ float4 XT[];  // per-wavefront store staging, kSlice each (sized at launch)
    const uint32_t lane = threadIdx.x & (kWave - 1);
    const int w = (int)(threadIdx.x / kWave);
    const int d = A.d, k = A.k;
    const int c0 = w * kChunk + (int)lane * 8;
    const bool act = c0 < d;
    const bool dword3 = (d & 31) == 0;
    const int grp_a = c0 >> A.lg_a, grp_q = c0 >> A.lg_q;
    const uint32_t ngq = (uint32_t)d >> A.lg_q, nga = (uint32_t)d >> A.lg_a;
    const uint32_t sh_fixed = (A.fixed && act) ? step_roundup(A.steps[grp_q]) : 0u;
    constexpr bool OUTL = OM == 1;
    const int32_t rix = load_ref_rows_v(A, lane);  // store rows of the gathered reference
    const int32_t fix = first_ref_index(A);        // and of the first row
    // per-group outliers: entries per row, this chunk's first entry and count
    const uint32_t gent = (uint32_t)k * ngq;
    const uint32_t gfirst = ((uint32_t)(w * kChunk) >> A.lg_q) * (uint32_t)k;
    const uint32_t gcount = ((uint32_t)__builtin_elementwise_min(kChunk, d - w * kChunk) >> A.lg_q) * (uint32_t)k;

    // inputs of one row for this lane: ref words, packed codes, coefficient
    // pair, scale, and either (lanes < k) one per-token outlier entry or
    // entries l and l + 64 of the chunk's per-group outliers
    struct In {
        uint4 rv;
        uint32_t lo, hi, cf, sh, ent, ent2;
    };
    // (zeros past the last row and past the end of the row; entries of lanes
    // >= k are never read)
    const uint32_t crb = (uint32_t)A.code_row_bytes;
    auto load = [&](uint32_t rw, int32_t ix) {
        const bool in_range = rw < A.tokens;
        const uint64_t r = (uint64_t)(in_range ? rw : 0);
        In in;
        in.rv = bload128(ref_row(A, rw, in_range, ix), (uint32_t)c0 * 2u);
        in.cf = bload32(rsrc(A.coef, r * nga, in_range ? nga * 4u : 0u), (uint32_t)grp_a * 4u);
        in.sh = bload16(rsrc(A.scale, r * ngq, (in_range && !A.fixed) ? ngq * 2u : 0u), (uint32_t)grp_q * 2u);
        if (A.fixed) in.sh = sh_fixed;
        load_codes<BITS>(rsrc(A.codes, r * crb, in_range ? crb : 0u), w, lane, dword3, in.lo, in.hi);
        in.ent = OUTL ? bload32(rsrc(A.outl, r * (uint64_t)k, in_range ? (uint32_t)k * 4u : 0u), lane * 4u) : 0u;
        in.ent2 = 0u;
        if constexpr (OM == 2) {
            const Rsrc rv = rsrc(A.gval, r * gent, in_range ? gent * 2u : 0u);
            const Rsrc ro = rsrc(A.goff, r * gent, in_range ? gent : 0u);
            const bool in0 = lane < gcount, in1 = lane + kWave < gcount;
            in.ent = bload16(rv, in0 ? (gfirst + lane) * 2u : kOut) | (bload8(ro, in0 ? gfirst + lane : kOut) << 16);
            in.ent2 = bload16(rv, in1 ? (gfirst + lane + kWave) * 2u : kOut) |
                      (bload8(ro, in1 ? gfirst + lane + kWave : kOut) << 16);
        }
        return in;
    };

    // One row: outliers of this chunk (lane i < k holds entry i) take R~ +
    // value, R~ formed from the channel's ref value and coefficient pair.
    // These are gathered first (just read by the owning lanes, so the reads
    // hit in cache), then the next-but-one row is prefetched into `nx`, so
    // waiting for the gathers does not wait for the prefetch.
    auto row_body = [&](const In& in, uint32_t row, uint32_t n, In& nx, uint32_t nrow) {
        const uint32_t ech = in.ent & 0xFFFFu;
        const bool pch = OUTL & (lane < (uint32_t)k) & (ech < (uint32_t)d) & ((ech >> 9) == (uint32_t)w);
        uint32_t gref = 0u, gcf = 0u;
        if constexpr (OUTL) {
            gref = bload16(ref_row(A, row, true, ref_index_v(A, rix, n)), pch ? ech * 2u : kOut);
            gcf = bload32(rsrc(A.coef, (uint64_t)row * nga, nga * 4u), pch ? (ech >> A.lg_a) * 4u : kOut);
        }
        nx = load(nrow, ref_index_v(A, rix, n + 1u));
        const float a = f16_wire(in.cf & 0xFFFFu), b0 = f16_wire(in.cf >> 16);
        const float s = f16_wire(in.sh);
        float r[8], rt[8], H[8];
        widen8(in.rv, r);
#pragma unroll
        for (int j = 0; j < 8; ++j) {  // R~ + q*s, q*s exact
            rt[j] = __builtin_fmaf(a, r[j], b0);
            H[j] = __builtin_fmaf((float)code_at<BITS>(in.lo, in.hi, j), s, rt[j]);
        }
        if constexpr (OM == 2) {
            // the k_g entries of this lane's group, pulled from the lanes that
            // loaded them; an entry whose offset falls in this lane's 8
            // channels replaces that channel by R~ + value
            const uint32_t lv = (uint32_t)A.lane_lv_q;
            const uint32_t mine = lane & ((1u << lv) - 1u), gbase = (lane >> lv) * (uint32_t)k;
            for (int i = 0; i < k; ++i) {
                const uint32_t src = gbase + (uint32_t)i;
                const int addr = (int)((src & (kWave - 1u)) << 2);
                const uint32_t e0 = (uint32_t)__builtin_amdgcn_ds_bpermute(addr, (int)in.ent);
                const uint32_t e1 = (uint32_t)__builtin_amdgcn_ds_bpermute(addr, (int)in.ent2);
                const uint32_t ent = src < (uint32_t)kWave ? e0 : e1;
                const uint32_t off = (ent >> 16) & 0xFFu;
                const float v = f16_wire(ent & 0xFFFFu);
                const bool here = (off >> 3) == mine;
#pragma unroll
                for (int j = 0; j < 8; ++j) H[j] = (here & ((off & 7u) == (uint32_t)j)) ? rt[j] + v : H[j];
            }
        }
        float4* st = XT + w * kSlice;
        put8(st, lane, H);
        wave_lds_sync();
        if (pch) {
            const float rt = __builtin_fmaf(f16_wire(gcf & 0xFFFFu), bf16_lo(gref), f16_wire(gcf >> 16));
            reinterpret_cast<float*>(st)[slice_float(ech & (uint32_t)(kChunk - 1))] = rt + f16_wire(in.ent >> 16);
        }
        wave_lds_sync();
        emit_xhat_flat(xhat_row(A, row), BF16, (uint32_t)(w * kChunk), lane, st);
    };

    // Rows in strides of the grid, two per iteration through two input
    // buffers (p holds the row being processed while q loads the next one, then
    // the roles swap), so no prefetched register is copied and nothing waits
    // for a prefetch before its row starts.
    const uint32_t G = gridDim.x;
    uint32_t row = blockIdx.x;
    In p = load(row, fix), q;
    // (a store that the range check drops, so that stores are outstanding at
    // the loop entry as at the end of every row; the compiler's wait analysis
    // then keeps later waits exact instead of waiting for everything)
    bstore32(rsrc(A.coef, 0, 0u), kOut, 0u);
    for (uint32_t n = 0; row < A.tokens; row += 2u * G, n += 2u) {
        row_body(p, row, n, q, row + G);
        if (row + G >= A.tokens) break;
        row_body(q, row + G, n + 1u, p, row + 2u * G);
    }
}

// ---------------------------------------------------------------------------
// Fit pooled over segments of rows (the affine-fit equation over all fitting
// positions of a segment).  Three launches: the per-(row, group) centred
// moments, their merge over each segment, then the encode with the merged
// pair of every row given.

struct Mom {
    float n, mr, mx, crr, crx;
};

// Pairwise merge of the centred moments of two disjoint sets (Chan, Golub and
// LeVeque), each step one rounded operation in a fixed order.
__device__ __forceinline__ Mom mom_merge(const Mom& a, const Mom& b) {
    const float n = a.n + b.n;
    const float dr = b.mr - a.mr, dx = b.mx - a.mx;
    const float fb = b.n / n;
    const float w = (a.n * b.n) / n;
    Mom m;
    m.n = n;
    m.mr = a.mr + dr * fb;
    m.mx = a.mx + dx * fb;
    m.crr = (a.crr + b.crr) + (dr * dr) * w;
    m.crx = (a.crx + b.crx) + (dr * dx) * w;
    return m;
}

// Moments of every (row, alignment group), as the per-token fit computes
// them: one workgroup per row (strided), one wavefront per 512-channel chunk,
// groups inside a chunk.  Written as float4 (m_r, m_x, C_rr, C_rx) to `mom`
// [T][d/g_a] (the wire's code section, which the encode overwrites later).
template <int GA>
__global__ __launch_bounds__(kWave * kMaxWaves) void rac_moments_kernel(Args A, float4* mom) {
    const uint32_t lane = threadIdx.x & (kWave - 1);
    const int w = (int)(threadIdx.x / kWave);
    const int d = A.d;
    const int c0 = w * kChunk + (int)lane * 8;
    const int lv_a = GA >= 0 ? GA : A.lane_lv_a;
    const bool first_a = (lane & ((1u << lv_a) - 1u)) == 0u;
    const uint32_t nga = (uint32_t)d >> A.lg_a, grp_a = (uint32_t)c0 >> A.lg_a;
    const uint32_t row_bytes = (uint32_t)d * 2u;
    for (uint32_t row = blockIdx.x; row < A.tokens; row += gridDim.x) {
        const uint64_t o = (uint64_t)row * (uint64_t)d;
        const uint4 xv = bload128(rsrc(A.x, o, row_bytes), (uint32_t)c0 * 2u);
        const uint4 rv = bload128(rsrc(A.ref, o, A.ref ? row_bytes : 0u), (uint32_t)c0 * 2u);
        float r[8], x[8], uu[8], uv[8];
        widen8(rv, r);
        widen8(xv, x);
        const float mr = lsum<GA>(tree8(r), lv_a) * A.inv_ga;
        const float mx = lsum<GA>(tree8(x), lv_a) * A.inv_ga;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float u = r[j] - mr, v = x[j] - mx;
            uu[j] = u * u;
            uv[j] = u * v;
        }
        const float crr = lsum<GA>(tree8(uu), lv_a);
        const float crx = lsum<GA>(tree8(uv), lv_a);
        if (first_a && c0 < d) mom[(uint64_t)row * nga + grp_a] = make_float4(mr, mx, crr, crx);
    }
}

// One workgroup of kPoolWaves wavefronts per (segment, alignment group)
// (beyond the largest grid one dispatch holds, workgroups take further pairs
// in strides of the grid):
// merges the segment's row moments over the binary-decomposition tree (a
// range of n rows splits into its first p rows, p the largest power of two
// below n, and the rest).  Rows are taken in blocks of 64, one block per
// wavefront at a time: inside a block, a bottom-up tree across lanes (an
// unpaired last element passes up), which is that tree for the block.  The
// pass's blocks (all whole but possibly the last) are merged the same way by
// the lanes of the first wavefront, which is again that tree over their rows.
// One thread takes the pass results in row order onto a stack of
// power-of-two sizes, merging whenever the top two are equal, and merges the
// stack from the top down at the end.  The fp16 pair goes to the coefficient
// slot of every row of the segment.  Segment bounds are clamped to [0, T], so no access leaves the buffers
// whatever the starts hold.
constexpr int kPoolWaves = 16;

__global__ __launch_bounds__(kWave * kPoolWaves) void rac_pool_kernel(Args A, const float4* mom) {
    __shared__ Mom blk[kPoolWaves];
    __shared__ uint32_t bsz[kPoolWaves];
    __shared__ Mom stk[40];
    __shared__ uint32_t ssz[40];
    __shared__ uint32_t cf_shared;
    const uint32_t lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
    const uint32_t nga = (uint32_t)A.d >> A.lg_a;
    const uint32_t pairs = (uint32_t)A.segments * nga;  // < 2^31
    const int64_t T = (int64_t)A.tokens;
    const float gn = (float)(1 << A.lg_a);
    // bottom-up tree over the first m lanes' moments (result in lane 0)
    auto lane_tree = [&](Mom v, uint32_t m, int levels) {
        for (int k = 0; k < levels; ++k) {
            const uint32_t off = 1u << k;
            const int addr = (int)(((lane + off) & (kWave - 1)) << 2);
            Mom p;
            p.n = __int_as_float(__builtin_amdgcn_ds_bpermute(addr, __float_as_int(v.n)));
            p.mr = __int_as_float(__builtin_amdgcn_ds_bpermute(addr, __float_as_int(v.mr)));
            p.mx = __int_as_float(__builtin_amdgcn_ds_bpermute(addr, __float_as_int(v.mx)));
            p.crr = __int_as_float(__builtin_amdgcn_ds_bpermute(addr, __float_as_int(v.crr)));
            p.crx = __int_as_float(__builtin_amdgcn_ds_bpermute(addr, __float_as_int(v.crx)));
            if ((lane & (2u * off - 1u)) == 0u && lane + off < m) v = mom_merge(v, p);
        }
        return v;
    };
    for (uint32_t pair = blockIdx.x; pair < pairs; pair += gridDim.x) {
        const uint32_t s = pair / nga, j = pair % nga;
        int64_t lo = A.seg_start[s], hi = A.seg_start[s + 1];
        lo = lo < 0 ? 0 : (lo > T ? T : lo);
        hi = hi < lo ? lo : (hi > T ? T : hi);
        int top = 0;  // (thread 0's)
        for (int64_t p0 = lo; p0 < hi; p0 += (int64_t)kWave * kPoolWaves) {
            const int64_t b0 = p0 + (int64_t)wv * kWave;
            const int64_t left = hi - b0;
            const uint32_t m = left <= 0 ? 0u : (left < kWave ? (uint32_t)left : (uint32_t)kWave);
            Mom v{0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
            if (lane < m) {
                const float4 f = mom[(uint64_t)(b0 + lane) * nga + j];
                v = Mom{gn, f.x, f.y, f.z, f.w};
            }
            v = lane_tree(v, m, 6);
            if (lane == 0u) {
                blk[wv] = v;
                bsz[wv] = m;
            }
            __syncthreads();
            if (wv == 0u) {
                // the pass's blocks: whole 64-row blocks, possibly a partial last one
                uint32_t nb = 0u, rows = 0u;
                for (int b = 0; b < kPoolWaves; ++b) {
                    nb += bsz[b] != 0u ? 1u : 0u;
                    rows += bsz[b];
                }
                Mom u{0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
                if (lane < nb) u = blk[lane];
                u = lane_tree(u, nb, 4);
                if (lane == 0u) {
                    stk[top] = u;
                    ssz[top] = rows;
                    ++top;
                    while (top >= 2 && ssz[top - 1] == ssz[top - 2]) {
                        stk[top - 2] = mom_merge(stk[top - 2], stk[top - 1]);
                        ssz[top - 2] *= 2u;
                        --top;
                    }
                }
            }
            __syncthreads();
        }
        if (threadIdx.x == 0u) {
            uint32_t cf = 0u;
            if (top > 0) {
                Mom r = stk[top - 1];
                for (int i = top - 2; i >= 0; --i) r = mom_merge(stk[i], r);
                cf = fit_coef(r.crr, r.crx, r.mr, r.mx);
            }
            cf_shared = cf;
        }
        __syncthreads();
        const uint32_t cf = cf_shared;
        if (A.pool_first_rows) {
            // the outlier encode takes the pair from the segment's first row and
            // writes every row's slot itself (4-byte stores from each segment's
            // 32 or more workgroups into shared lines cost 4 us here)
            if (threadIdx.x == 0u && lo < hi) bstore32(rsrc(A.coef, (uint64_t)lo * nga, nga * 4u), j * 4u, cf);
        } else {
            for (int64_t t = lo + threadIdx.x; t < hi; t += (int64_t)kWave * kPoolWaves)
                bstore32(rsrc(A.coef, (uint64_t)t * nga, nga * 4u), j * 4u, cf);
        }
        __syncthreads();  // the next pair reuses the shared state
    }
}

// ---------------------------------------------------------------------------
// Reconstruction error of a coded sample (the offline calibration's quality
// measure): sum (x - H-hat)^2, sum x^2 and max |x - H-hat| in binary64.
// Every difference is one binary64 subtraction of the exact widened values,
// every square one rounded multiply.  The sums have a fixed order whatever
// the device: block b takes rows [8b, 8b + 8), thread t its 8-element pieces
// t, t + 256, ... in sequence, then a pairwise tree over the 256 threads
// gives the block's partial; a single block reduces the partials the same
// way (thread t: partials t, t + 256, ..., then the tree).

constexpr int kErrRows = 8;         // token rows per partial
constexpr int kErrThreads = 256;

struct ErrSums {
    double se, sx, mx;
};

__device__ __forceinline__ ErrSums err_tree(ErrSums v, double (*sh)[kErrThreads]) {
    const uint32_t t = threadIdx.x;
    sh[0][t] = v.se;
    sh[1][t] = v.sx;
    sh[2][t] = v.mx;
    __syncthreads();
    for (uint32_t s = kErrThreads / 2; s > 0; s >>= 1) {
        if (t < s) {
            sh[0][t] = sh[0][t] + sh[0][t + s];
            sh[1][t] = sh[1][t] + sh[1][t + s];
            sh[2][t] = __builtin_fmax(sh[2][t], sh[2][t + s]);
        }
        __syncthreads();
    }
    return ErrSums{sh[0][0], sh[1][0], sh[2][0]};
}

__global__ __launch_bounds__(kErrThreads) void rac_error_kernel(const uint16_t* x, const void* xhat, int32_t bf16,
                                                                uint32_t tokens, int32_t d, double* part) {
    __shared__ double sh[3][kErrThreads];
    const uint32_t parts = (uint32_t)(((uint64_t)tokens + kErrRows - 1) / kErrRows);
    // (beyond the largest grid one dispatch holds, blocks take further parts
    // in strides of the grid; each part's sum is the same either way)
    for (uint32_t pt = blockIdx.x; pt < parts; pt += gridDim.x) {
        const uint64_t row0 = (uint64_t)pt * kErrRows;
        const uint64_t rows = tokens - row0 < (uint64_t)kErrRows ? tokens - row0 : (uint64_t)kErrRows;
        const uint64_t base = row0 * (uint64_t)d, n = rows * (uint64_t)d;  // n is a multiple of 8
        ErrSums v{0.0, 0.0, 0.0};
        for (uint64_t e = (uint64_t)threadIdx.x * 8u; e < n; e += (uint64_t)kErrThreads * 8u) {
            float xf[8], hf[8];
            widen8(*reinterpret_cast<const uint4*>(x + base + e), xf);
            if (bf16) {
                widen8(*reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(xhat) + base + e), hf);
            } else {
                const float4* hp = reinterpret_cast<const float4*>(static_cast<const float*>(xhat) + base + e);
                const float4 a = hp[0], b = hp[1];
                hf[0] = a.x; hf[1] = a.y; hf[2] = a.z; hf[3] = a.w;
                hf[4] = b.x; hf[5] = b.y; hf[6] = b.z; hf[7] = b.w;
            }
    #pragma unroll
            for (int j = 0; j < 8; ++j) {
                const double xv = (double)xf[j];
                const double dd = xv - (double)hf[j];
                v.se = v.se + dd * dd;
                v.sx = v.sx + xv * xv;
                v.mx = __builtin_fmax(v.mx, __builtin_fabs(dd));
            }
        }
        const ErrSums r = err_tree(v, sh);
        if (threadIdx.x == 0) {
            part[3u * pt + 0u] = r.se;
            part[3u * pt + 1u] = r.sx;
            part[3u * pt + 2u] = r.mx;
        }
        __syncthreads();  // the next part reuses sh
    }
}

__global__ __launch_bounds__(kErrThreads) void rac_error_final_kernel(const double* part, uint32_t nparts,
                                                                      double* out) {
    __shared__ double sh[3][kErrThreads];
    ErrSums v{0.0, 0.0, 0.0};
    for (uint32_t p = threadIdx.x; p < nparts; p += kErrThreads) {
        v.se = v.se + part[3u * p + 0u];
        v.sx = v.sx + part[3u * p + 1u];
        v.mx = __builtin_fmax(v.mx, part[3u * p + 2u]);
    }
    const ErrSums r = err_tree(v, sh);
    if (threadIdx.x == 0) {
        out[0] = r.se;
        out[1] = r.sx;
        out[2] = r.mx;
    }
}

}  // namespace

// The allocation-free variant of the error reduction keeps its partials in
// this array instead of a caller workspace: one copy per device, held until
// the process ends.  Host code never uses the name itself (on the host it is
// only a stand-in for the device symbol); it uses the device address that
// hipGetSymbolAddress gives for the current device.
constexpr uint32_t kScratchParts = 16384;  // partials of 8 rows: up to 131072 token rows
static __device__ __align__(256) double scratch[3 * kScratchParts];

namespace {

// ---------------------------------------------------------------------------
// Host side

bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }
int ilog2(int64_t v) { int l = 0; while ((int64_t(1) << l) < v) ++l; return l; }
uint64_t up256(uint64_t v) { return (v + 255u) & ~uint64_t(255); }

bool config_valid(const rac_config* c) {
    if (!c) return false;
    if (c->tokens < 0 || c->tokens > 0x7FFFFFFFll) return false;
    if (c->hidden < 8 || c->hidden > 65535 || c->hidden % 8 != 0) return false;
    if (!is_pow2(c->group_align) || c->group_align < 8 || c->group_align > c->hidden ||
        c->hidden % c->group_align != 0)
        return false;
    if (!is_pow2(c->group_quant) || c->group_quant < 8 || c->group_quant > c->hidden ||
        c->hidden % c->group_quant != 0)
        return false;
    if (c->bits != 2 && c->bits != 3 && c->bits != 4 && c->bits != 8) return false;
    if (c->flags & ~uint32_t(RAC_FLAG_FIXED_STEP | RAC_FLAG_XHAT_BF16 | RAC_FLAG_GROUP_OUTLIERS |
                             RAC_FLAG_LAUNCH_STRIDED | RAC_FLAG_LAUNCH_PER_ROW))
        return false;
    if ((c->flags & RAC_FLAG_LAUNCH_STRIDED) && (c->flags & RAC_FLAG_LAUNCH_PER_ROW)) return false;
    if (c->flags & RAC_FLAG_GROUP_OUTLIERS) {
        if (c->group_quant > 256) return false;  // u8 in-group offsets
        if (c->outlier_k < 1 || c->outlier_k > 16 || c->outlier_k > c->group_quant / 4) return false;
    } else if (c->outlier_k < 0 || c->outlier_k > 64 || c->outlier_k > c->hidden) {
        return false;
    }
    return true;
}

bool grouped(const rac_config* c) { return (c->flags & RAC_FLAG_GROUP_OUTLIERS) != 0; }

struct Sizes {
    rac_layout L;
    uint64_t coef, scale, codes, outl, ooff;
};

Sizes sizes_of(const rac_config* c) {
    Sizes s;
    const uint64_t T = (uint64_t)c->tokens, d = (uint64_t)c->hidden;
    s.coef = T * (d / (uint64_t)c->group_align) * 4u;
    s.scale = (c->flags & RAC_FLAG_FIXED_STEP) ? 0u : T * (d / (uint64_t)c->group_quant) * 2u;
    s.codes = T * d * (uint64_t)c->bits / 8u;
    const uint64_t gent = T * (d / (uint64_t)c->group_quant) * (uint64_t)c->outlier_k;
    s.outl = grouped(c) ? gent * 2u : T * (uint64_t)c->outlier_k * 4u;
    s.ooff = grouped(c) ? gent : 0u;
    s.L.off_coef = 256;
    s.L.off_scale = up256(s.L.off_coef + s.coef);
    s.L.off_codes = up256(s.L.off_scale + s.scale);
    s.L.off_outl = up256(s.L.off_codes + s.codes);
    s.L.off_ooff = grouped(c) ? up256(s.L.off_outl + s.outl) : 0u;
    s.L.total = grouped(c) ? up256(s.L.off_ooff + s.ooff) : up256(s.L.off_outl + s.outl);
    return s;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

Args make_args(const rac_config* c, const Sizes& S) {
    Args A{};
    A.off_scale = S.L.off_scale;
    A.off_codes = S.L.off_codes;
    A.off_outl = S.L.off_outl;
    A.total = S.L.total;
    // without per-group outliers the offset array is empty, at the end
    A.off_ooff = grouped(c) ? S.L.off_ooff : S.L.total;
    A.end_ooff = A.off_ooff + S.ooff;
    A.end_coef = S.L.off_coef + S.coef;
    A.end_scale = S.L.off_scale + S.scale;
    A.end_codes = S.L.off_codes + S.codes;
    A.end_outl = S.L.off_outl + S.outl;
    A.code_row_bytes = c->hidden * c->bits / 8;
    A.tokens = (uint32_t)c->tokens;
    A.d = c->hidden;
    A.nch = (c->hidden + kChunk - 1) / kChunk;
    A.lg_a = ilog2(c->group_align);
    A.lg_q = ilog2(c->group_quant);
    A.lane_lv_a = ilog2(c->group_align >= kChunk ? kChunk / 8 : c->group_align / 8);
    A.lane_lv_q = ilog2(c->group_quant >= kChunk ? kChunk / 8 : c->group_quant / 8);
    A.lg_cpg_a = c->group_align > kChunk ? ilog2(c->group_align / kChunk) : 0;
    A.lg_cpg_q = c->group_quant > kChunk ? ilog2(c->group_quant / kChunk) : 0;
    A.k = c->outlier_k;
    A.gout = grouped(c) ? 1 : 0;
    A.fixed = (c->flags & RAC_FLAG_FIXED_STEP) ? 1 : 0;
    A.xhat_bf16 = (c->flags & RAC_FLAG_XHAT_BF16) ? 1 : 0;
    A.inv_ga = 1.0f / (float)c->group_align;
    A.launch_shape = (c->flags & RAC_FLAG_LAUNCH_STRIDED) ? 1 : (c->flags & RAC_FLAG_LAUNCH_PER_ROW) ? 2 : 0;
    return A;
}

void set_sections(Args& A, const Sizes& S) {
    A.coef = reinterpret_cast<uint32_t*>(A.wire + S.L.off_coef);
    A.scale = reinterpret_cast<uint16_t*>(A.wire + S.L.off_scale);
    A.codes = A.wire + S.L.off_codes;
    A.outl = reinterpret_cast<uint32_t*>(A.wire + S.L.off_outl);
    A.gval = reinterpret_cast<uint16_t*>(A.wire + S.L.off_outl);
    A.goff = A.wire + (A.gout ? S.L.off_ooff : S.L.total);
}

void fill_header(Args& A, const rac_config* c, bool zero_ref, bool pooled = false) {
    uint8_t h[96] = {0};
    auto put16 = [&](int o, uint32_t v) { h[o] = (uint8_t)v; h[o + 1] = (uint8_t)(v >> 8); };
    auto put32 = [&](int o, uint32_t v) { for (int i = 0; i < 4; ++i) h[o + i] = (uint8_t)(v >> (8 * i)); };
    auto put64 = [&](int o, uint64_t v) { for (int i = 0; i < 8; ++i) h[o + i] = (uint8_t)(v >> (8 * i)); };
    uint32_t flags = 0;
    if (c->outlier_k > 0 && !grouped(c)) flags |= 1u;
    if (c->flags & RAC_FLAG_FIXED_STEP) flags |= 2u;
    if (zero_ref) flags |= 4u;
    if (grouped(c)) flags |= 8u;
    if (pooled) flags |= 16u;
    put32(0, 0x31434152u);
    put16(4, 2u);
    put16(6, flags);
    put32(8, (uint32_t)c->tokens);
    put32(12, (uint32_t)c->hidden);
    put32(16, (uint32_t)c->group_align);
    put32(20, (uint32_t)c->group_quant);
    h[24] = (uint8_t)c->bits;
    h[25] = 1;
    h[26] = (c->flags & RAC_FLAG_FIXED_STEP) ? 0 : 1;
    h[27] = grouped(c) ? 2 : (c->outlier_k > 0 ? 1 : 0);
    put16(28, (uint32_t)c->outlier_k);
    put64(32, (uint64_t)256);
    put64(40, A.off_scale);
    put64(48, A.off_codes);
    put64(56, A.off_outl);
    put64(64, A.total);
    put64(72, grouped(c) ? A.off_ooff : 0u);
    for (int i = 0; i < 24; ++i)
        A.hdr[i] = (uint32_t)h[4 * i] | ((uint32_t)h[4 * i + 1] << 8) | ((uint32_t)h[4 * i + 2] << 16) |
                   ((uint32_t)h[4 * i + 3] << 24);
}

using KernelFn = void (*)(Args);

template <int GA, int GQ, int OM>
KernelFn encode_for_bits(int bits) {
    switch (bits) {
        case 2: return rac_encode_kernel<2, GA, GQ, OM>;
        case 3: return rac_encode_kernel<3, GA, GQ, OM>;
        case 4: return rac_encode_kernel<4, GA, GQ, OM>;
        default: return rac_encode_kernel<8, GA, GQ, OM>;
    }
}

// (groups spanning chunks, GQ = 7, exceed the 256 channels of per-group
// outliers, so that form has no mode 2)
template <int GA, int GQ>
KernelFn encode_for(int bits, int om) {
    if constexpr (GQ != 7) {
        if (om == 2) return encode_for_bits<GA, GQ, 2>(bits);
    }
    return om == 1 ? encode_for_bits<GA, GQ, 1>(bits) : encode_for_bits<GA, GQ, 0>(bits);
}

int outlier_mode(const Args& A) { return A.gout ? 2 : (A.k > 0 ? 1 : 0); }

// Specialized group shapes: 64/64, 128/128, the mixed 64/128 and 128/64, and
// 128 with one scale per row of up to 8192 channels; anything else takes the
// generic kernel.
KernelFn pick_encode(const Args& A, int bits) {
    const int ga = A.lg_cpg_a > 0 ? 7 : A.lane_lv_a;
    const int gq = A.lg_cpg_q > 0 ? 7 : A.lane_lv_q;
    const int om = outlier_mode(A);
    if (ga == 3 && gq == 3) return encode_for<3, 3>(bits, om);
    if (ga == 4 && gq == 4) return encode_for<4, 4>(bits, om);
    if (ga == 3 && gq == 4) return encode_for<3, 4>(bits, om);
    if (ga == 4 && gq == 3) return encode_for<4, 3>(bits, om);
    if (ga == 4 && gq == 7) return encode_for<4, 7>(bits, om);
    return encode_for<-1, -1>(bits, om);
}

template <int GA, int GQ, int CPW, bool GIVEN, bool TWO, bool BIG>
KernelFn rows_for_bits(int bits) {
    switch (bits) {
        case 2: return rac_encode_rows_kernel<2, GA, GQ, kRowsWaves, CPW, GIVEN, TWO, BIG>;
        case 3: return rac_encode_rows_kernel<3, GA, GQ, kRowsWaves, CPW, GIVEN, TWO, BIG>;
        case 4: return rac_encode_rows_kernel<4, GA, GQ, kRowsWaves, CPW, GIVEN, TWO, BIG>;
        default: return rac_encode_rows_kernel<8, GA, GQ, kRowsWaves, CPW, GIVEN, TWO, BIG>;
    }
}

template <int GA, int GQ, int CPW, bool GIVEN>
KernelFn rows_for_cpw(int bits, int k) {
    if constexpr (GIVEN) {
        return rows_for_bits<GA, GQ, CPW, true, false, false>(bits);
    } else {
        if (k > kTop2) return rows_for_bits<GA, GQ, CPW, false, false, true>(bits);
        if (k > kTop1) return rows_for_bits<GA, GQ, CPW, false, true, false>(bits);
        return rows_for_bits<GA, GQ, CPW, false, false, false>(bits);
    }
}

// Rows of up to 4096 channels: two chunks per wavefront; up to 8192: four.
// The two-value threshold for kTop1 < k <= kTop2, and with the larger
// candidate list beyond (not with given pairs, which keep the one-value
// bound and the smaller list: every bound and list size is exact).
template <int GA, int GQ, bool GIVEN = false>
KernelFn rows_for(int bits, int d, int k) {
    if (d <= kRowsWaves * 2 * kChunk) return rows_for_cpw<GA, GQ, 2, GIVEN>(bits, k);
    return rows_for_cpw<GA, GQ, 4, GIVEN>(bits, k);
}

// Rows with outliers take the NW-wavefront kernel when it holds the whole
// row and both group sizes fit in a chunk (calibrated step tables take the
// one-wavefront-per-chunk kernel).
bool use_rows_kernel(const Args& A) {
    return outlier_mode(A) == 1 && !A.fixed && A.d <= kRowsMaxD && A.lg_cpg_a == 0 && A.lg_cpg_q == 0;
}

KernelFn pick_rows(const Args& A, int bits) {
    // given pairs (pooled fit): the fixed 128 and 64 shapes and the generic one
    if (A.cf_given) {
        if (A.lane_lv_a == 4 && A.lane_lv_q == 4) return rows_for<4, 4, true>(bits, A.d, A.k);
        if (A.lane_lv_a == 3 && A.lane_lv_q == 3) return rows_for<3, 3, true>(bits, A.d, A.k);
        return rows_for<-1, -1, true>(bits, A.d, A.k);
    }
    if (A.lane_lv_a == 3 && A.lane_lv_q == 3) return rows_for<3, 3>(bits, A.d, A.k);
    if (A.lane_lv_a == 4 && A.lane_lv_q == 4) return rows_for<4, 4>(bits, A.d, A.k);
    if (A.lane_lv_a == 3 && A.lane_lv_q == 4) return rows_for<3, 4>(bits, A.d, A.k);
    if (A.lane_lv_a == 4 && A.lane_lv_q == 3) return rows_for<4, 3>(bits, A.d, A.k);
    return rows_for<-1, -1>(bits, A.d, A.k);
}

template <int OM, bool BF16>
KernelFn decode_for(int bits) {
    switch (bits) {
        case 2: return rac_decode_kernel<2, OM, BF16>;
        case 3: return rac_decode_kernel<3, OM, BF16>;
        case 4: return rac_decode_kernel<4, OM, BF16>;
        default: return rac_decode_kernel<8, OM, BF16>;
    }
}

KernelFn pick_decode(const Args& A, int bits) {
    const bool bf16 = A.xhat_bf16 != 0;
    switch (outlier_mode(A)) {
        case 1: return bf16 ? decode_for<1, true>(bits) : decode_for<1, false>(bits);
        case 2: return bf16 ? decode_for<2, true>(bits) : decode_for<2, false>(bits);
        default: return bf16 ? decode_for<0, true>(bits) : decode_for<0, false>(bits);
    }
}

// Launch facts of one kernel on one device: compute units and resident
// workgroups per compute unit at a block size and dynamic LDS size.  They do
// not change while the process runs, so each is queried once and kept in a
// fixed table (no host or device allocation); a full table only means that
// later combinations are queried on every launch.
struct Occupancy {
    const void* fn;
    int dev, threads;
    size_t lds;
    int cus, per_cu;
};
constexpr int kOccSlots = 256;
Occupancy g_occ[kOccSlots];
int g_occ_used = 0;
std::mutex g_occ_mu;

rac_status resident(const void* fn, int threads, size_t lds, int* cus, int* per_cu) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return RAC_ERR_HIP;
    {
        std::lock_guard<std::mutex> lock(g_occ_mu);
        for (int i = 0; i < g_occ_used; ++i) {
            const Occupancy& o = g_occ[i];
            if (o.fn == fn && o.dev == dev && o.threads == threads && o.lds == lds) {
                *cus = o.cus;
                *per_cu = o.per_cu;
                return RAC_OK;
            }
        }
    }
    int c = 0, p = 0;
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        (fn && hipOccupancyMaxActiveBlocksPerMultiprocessor(&p, fn, threads, lds) != hipSuccess))
        return RAC_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_occ_mu);
    if (g_occ_used < kOccSlots) g_occ[g_occ_used++] = Occupancy{fn, dev, threads, lds, c, p};
    *cus = c;
    *per_cu = p;
    return RAC_OK;
}

// Compute units of the current device (cached like the occupancy).
rac_status device_cus(int* cus) {
    int unused = 0;
    return resident(nullptr, 0, 0, cus, &unused);
}

// One workgroup per token row.  Large row counts use a grid of as many
// workgroups as the device keeps resident (at most max_per_cu per compute
// unit), each taking rows in strides (and prefetching its next row); small
// counts, and counts that would give every resident workgroup more than
// kStridedRowsMax rows, launch one workgroup per row.  The launch flags of the
// configuration override that choice for more than 256 rows.  (Over many rows the
// strided workgroups drift apart, so the rows in flight spread over the
// tensors and the HBM writes lose locality; with one workgroup per row the
// dispatcher hands rows out in order as workgroups finish, which keeps them
// together.  Measured on a 65536 x 3584 tensor: 9% off the encode, 13% off
// the decode; at four rows per workgroup the two are even.)
rac_status launch(KernelFn fn, Args A, hipStream_t stream, int threads = 0, int max_per_cu = 0) {
    const int64_t rows = A.tokens;
    // kernels launched with one wavefront per chunk stage through a
    // dynamically sized slice per wavefront
    const bool staged = threads == 0;
    if (staged) threads = A.nch * kWave;
    const size_t lds = staged ? (size_t)A.nch * kSlice * sizeof(float4) : 0;
    int64_t blocks = rows <= 0 ? 1 : rows;
    if (rows > 256) {
        int cus = 0, per_cu = 0;
        if (resident(reinterpret_cast<const void*>(fn), threads, lds, &cus, &per_cu) != RAC_OK) return RAC_ERR_HIP;
        const int64_t fits = (int64_t)cus * (per_cu > 0 ? per_cu : 1);  // workgroups the device holds at once
        const bool strided = A.launch_shape == 1 || (A.launch_shape == 0 && rows <= kStridedRowsMax * fits);
        if (strided) {
            if (max_per_cu > 0 && per_cu > max_per_cu) per_cu = max_per_cu;
            int64_t resident = (int64_t)cus * (per_cu > 0 ? per_cu : 1);
            // a gathered reference: at most kMaxGatherRows rows per workgroup,
            // whose indices are loaded once up front
            const int64_t gather_min = (rows + kMaxGatherRows - 1) / kMaxGatherRows;
            if (A.ref_rows && resident < gather_min) resident = gather_min;
            if (blocks > resident) blocks = resident;
        }
    }
    // A dispatch holds fewer than 2^32 work-items per dimension: beyond that
    // the workgroups stride over the rows (every kernel takes rows in strides
    // of the grid).  A gathered reference allows at most kMaxGatherRows rows
    // per workgroup.
    const int64_t max_blocks = (int64_t)(kMaxDispatchItems / (uint32_t)threads);
    if (blocks > max_blocks) blocks = max_blocks;
    if (A.ref_rows && blocks * kMaxGatherRows < rows) return RAC_ERR_UNSUPPORTED;
    void* args[] = {&A};
    const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(fn), dim3((unsigned)blocks),
                                         dim3((unsigned)threads), args, lds, stream);
    return e == hipSuccess ? RAC_OK : RAC_ERR_HIP;
}

rac_status common_checks(const rac_config* cfg) {
    if (!config_valid(cfg)) return RAC_ERR_INVALID;
    if (cfg->hidden > kMaxWaves * kChunk) return RAC_ERR_UNSUPPORTED;
    return RAC_OK;
}

// A gathered reference: a store of store_rows rows and one int32 index per
// token row (NULL ref_rows: the reference is ref itself, one row per token).
rac_status check_gather(const void* store, int64_t store_rows, const int32_t* ref_rows, bool gather) {
    if (!gather) return RAC_OK;
    if (store_rows < 0 || store_rows > 0x7FFFFFFFll) return RAC_ERR_INVALID;
    if (store && !ref_rows) return RAC_ERR_INVALID;
    if (ref_rows && !aligned(ref_rows, 4)) return RAC_ERR_ALIGN;
    return RAC_OK;
}

rac_status run_decode(const rac_config* cfg, const void* wire, const void* ref, const float* steps,
                      void* xhat, hipStream_t stream, bool gather = false, int64_t store_rows = 0,
                      const int32_t* ref_rows = nullptr) {
    rac_status st = common_checks(cfg);
    if (st != RAC_OK) return st;
    if (!wire || (cfg->tokens > 0 && !xhat)) return RAC_ERR_INVALID;
    if ((cfg->flags & RAC_FLAG_FIXED_STEP) && !steps) return RAC_ERR_INVALID;
    if ((st = check_gather(ref, store_rows, ref_rows, gather)) != RAC_OK) return st;
    if (!aligned(wire, 256) || !aligned(xhat, 16) || (ref && !aligned(ref, 16)) ||
        (steps && !aligned(steps, 4)))
        return RAC_ERR_ALIGN;
    if (cfg->tokens == 0) return RAC_OK;
    const Sizes S = sizes_of(cfg);
    Args A = make_args(cfg, S);
    A.wire = const_cast<uint8_t*>(static_cast<const uint8_t*>(wire));
    set_sections(A, S);
    A.ref = static_cast<const uint16_t*>(ref);
    A.ref_rows = (gather && ref) ? ref_rows : nullptr;
    A.store_rows = (uint32_t)store_rows;
    A.steps = steps;
    A.xhat = xhat;
    // (with outliers, two workgroups per compute unit, each taking more rows,
    // measured fastest: 4-8% below a full grid at 4096 x 4096 and 16384 x 3584)
    return launch(pick_decode(A, cfg->bits), A, stream, 0, outlier_mode(A) == 1 ? 2 : 0);
}

}  // namespace

extern "C" {

rac_status rac_wire_layout(const rac_config* cfg, rac_layout* out) {
    if (!config_valid(cfg) || !out) return RAC_ERR_INVALID;
    *out = sizes_of(cfg).L;
    return RAC_OK;
}

rac_status rac_saturation_summary(const rac_config* cfg, const void* wire_host, size_t len, int64_t* rows,
                                  uint32_t* bits) {
    if (!config_valid(cfg) || !wire_host) return RAC_ERR_INVALID;
    const Sizes S = sizes_of(cfg);
    if (len < S.L.total) return RAC_ERR_INVALID;
    const uint8_t* w = static_cast<const uint8_t*>(wire_host);
    auto inf16 = [&](uint64_t off) { return ((w[off] | (w[off + 1] << 8)) & 0x7FFFu) == 0x7C00u; };
    const uint64_t T = (uint64_t)cfg->tokens, d = (uint64_t)cfg->hidden;
    const uint64_t nga = d / (uint64_t)cfg->group_align, ngq = d / (uint64_t)cfg->group_quant;
    const uint64_t k = (uint64_t)cfg->outlier_k;
    int64_t n = 0;
    uint32_t all = 0;
    for (uint64_t t = 0; t < T; ++t) {
        uint32_t r = 0;
        for (uint64_t j = 0; j < 2 * nga; ++j) r |= inf16(S.L.off_coef + (t * 2 * nga + j) * 2) ? 1u : 0u;
        if (!(cfg->flags & RAC_FLAG_FIXED_STEP))
            for (uint64_t j = 0; j < ngq; ++j) r |= inf16(S.L.off_scale + (t * ngq + j) * 2) ? 2u : 0u;
        if (grouped(cfg)) {
            for (uint64_t j = 0; j < ngq * k; ++j) r |= inf16(S.L.off_outl + (t * ngq * k + j) * 2) ? 4u : 0u;
        } else {
            for (uint64_t j = 0; j < k; ++j) r |= inf16(S.L.off_outl + (t * k + j) * 4 + 2) ? 4u : 0u;
        }
        n += r ? 1 : 0;
        all |= r;
    }
    if (rows) *rows = n;
    if (bits) *bits = all;
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
    if (g32(0) != 0x31434152u || g16(4) != 2u) return RAC_ERR_FORMAT;
    const uint32_t flags = g16(6);
    if (flags & ~31u) return RAC_ERR_FORMAT;
    if ((flags & 1u) && (flags & 8u)) return RAC_ERR_FORMAT;
    rac_config c{};
    c.tokens = g32(8);
    c.hidden = (int32_t)g32(12);
    c.group_align = (int32_t)g32(16);
    c.group_quant = (int32_t)g32(20);
    c.bits = h[24];
    c.outlier_k = (int32_t)g16(28);
    c.flags = ((flags & 2u) ? RAC_FLAG_FIXED_STEP : 0u) | ((flags & 8u) ? RAC_FLAG_GROUP_OUTLIERS : 0u);
    if (g32(12) > 65535u || g32(16) > 65535u || g32(20) > 65535u) return RAC_ERR_FORMAT;
    if (!config_valid(&c)) return RAC_ERR_FORMAT;
    if (!(flags & 8u) && ((flags & 1u) != 0) != (c.outlier_k > 0)) return RAC_ERR_FORMAT;
    const uint32_t ofmt = (flags & 8u) ? 2u : (c.outlier_k > 0 ? 1u : 0u);
    if (h[25] != 1 || h[26] != ((flags & 2u) ? 0 : 1) || h[27] != ofmt) return RAC_ERR_FORMAT;
    const Sizes S = sizes_of(&c);
    if (g64(32) != S.L.off_coef || g64(40) != S.L.off_scale || g64(48) != S.L.off_codes ||
        g64(56) != S.L.off_outl || g64(64) != S.L.total || g64(72) != S.L.off_ooff)
        return RAC_ERR_FORMAT;
    for (int i = 30; i < 32; ++i)
        if (h[i]) return RAC_ERR_FORMAT;
    for (int i = 80; i < 256; ++i)
        if (h[i]) return RAC_ERR_FORMAT;
    *out = c;
    if (zero_ref) *zero_ref = (flags & 4u) ? 1 : 0;
    return RAC_OK;
}

}  // extern "C"

namespace {

rac_status run_encode(const rac_config* cfg, const void* x, const void* ref, const float* fixed_steps,
                      void* wire, size_t wire_cap, void* xhat, hipStream_t stream, bool gather,
                      int64_t store_rows, const int32_t* ref_rows) {
    rac_status st = common_checks(cfg);
    if (st != RAC_OK) return st;
    if (!wire || (cfg->tokens > 0 && !x)) return RAC_ERR_INVALID;
    if ((cfg->flags & RAC_FLAG_FIXED_STEP) && !fixed_steps) return RAC_ERR_INVALID;
    if ((st = check_gather(ref, store_rows, ref_rows, gather)) != RAC_OK) return st;
    if (!aligned(wire, 256) || !aligned(x, 16) || (ref && !aligned(ref, 16)) ||
        (xhat && !aligned(xhat, 16)) || (fixed_steps && !aligned(fixed_steps, 4)))
        return RAC_ERR_ALIGN;
    const Sizes S = sizes_of(cfg);
    if (wire_cap < S.L.total) return RAC_ERR_CAPACITY;
    Args A = make_args(cfg, S);
    A.x = static_cast<const uint16_t*>(x);
    A.ref = static_cast<const uint16_t*>(ref);
    A.ref_rows = (gather && ref) ? ref_rows : nullptr;
    A.store_rows = (uint32_t)store_rows;
    A.steps = (cfg->flags & RAC_FLAG_FIXED_STEP) ? fixed_steps : nullptr;
    A.wire = static_cast<uint8_t*>(wire);
    set_sections(A, S);
    A.xhat = xhat;
    A.write_header = 1;
    fill_header(A, cfg, ref == nullptr);
    if (use_rows_kernel(A)) return launch(pick_rows(A, cfg->bits), A, stream, kRowsWaves * kWave);
    return launch(pick_encode(A, cfg->bits), A, stream);
}

}  // namespace

extern "C" {

rac_status rac_encode(const rac_config* cfg, const void* x, const void* ref, const float* fixed_steps,
                      void* wire, size_t wire_cap, void* xhat, rac_stream_t stream) {
    return run_encode(cfg, x, ref, fixed_steps, wire, wire_cap, xhat, stream, false, 0, nullptr);
}

rac_status rac_encode_gather(const rac_config* cfg, const void* x, const void* ref_store, int64_t store_rows,
                             const int32_t* ref_rows, const float* fixed_steps, void* wire, size_t wire_cap,
                             void* xhat, rac_stream_t stream) {
    return run_encode(cfg, x, ref_store, fixed_steps, wire, wire_cap, xhat, stream, true, store_rows, ref_rows);
}

rac_status rac_decode_gather(const rac_config* cfg, const void* wire, const void* ref_store, int64_t store_rows,
                             const int32_t* ref_rows, const float* fixed_steps, void* xhat, rac_stream_t stream) {
    return run_decode(cfg, wire, ref_store, fixed_steps, xhat, stream, true, store_rows, ref_rows);
}

rac_status rac_encode_pooled(const rac_config* cfg, const void* x, const void* ref, int64_t segments,
                             const int32_t* seg_start, const float* fixed_steps, void* wire, size_t wire_cap,
                             void* xhat, rac_stream_t stream) {
    rac_status st = common_checks(cfg);
    if (st != RAC_OK) return st;
    if (!wire || !x || cfg->tokens < 1 || !seg_start || segments < 1 || segments > cfg->tokens)
        return RAC_ERR_INVALID;
    if ((cfg->flags & RAC_FLAG_FIXED_STEP) && !fixed_steps) return RAC_ERR_INVALID;
    // groups inside a chunk; the row moments (16 B per row and group) fit in
    // the code section they are staged in
    if (cfg->group_align > kChunk || (int64_t)cfg->group_align * cfg->bits < 128) return RAC_ERR_UNSUPPORTED;
    if (!aligned(wire, 256) || !aligned(x, 16) || (ref && !aligned(ref, 16)) || (xhat && !aligned(xhat, 16)) ||
        (fixed_steps && !aligned(fixed_steps, 4)) || !aligned(seg_start, 4))
        return RAC_ERR_ALIGN;
    const Sizes S = sizes_of(cfg);
    if (wire_cap < S.L.total) return RAC_ERR_CAPACITY;
    // every check and device query before the first launch: a rejected call
    // leaves the wire untouched
    const uint64_t nga = (uint64_t)(cfg->hidden / cfg->group_align);
    const uint64_t pblocks = (uint64_t)segments * nga;
    if (pblocks > 0x7FFFFFFFull) return RAC_ERR_UNSUPPORTED;
    int cus = 0;
    if (device_cus(&cus) != RAC_OK) return RAC_ERR_HIP;
    Args A = make_args(cfg, S);
    A.x = static_cast<const uint16_t*>(x);
    A.ref = static_cast<const uint16_t*>(ref);
    A.steps = (cfg->flags & RAC_FLAG_FIXED_STEP) ? fixed_steps : nullptr;
    A.wire = static_cast<uint8_t*>(wire);
    set_sections(A, S);
    A.xhat = xhat;
    A.segments = (int32_t)segments;
    A.seg_start = seg_start;
    float4* mom = reinterpret_cast<float4*>(A.codes);
    A.pool_first_rows = use_rows_kernel(A) ? 1 : 0;
    // 1. row moments
    const int threads = A.nch * kWave;
    void* margs[] = {&A, &mom};
    const void* mfn = A.lane_lv_a == 3 ? reinterpret_cast<const void*>(rac_moments_kernel<3>)
                    : A.lane_lv_a == 4 ? reinterpret_cast<const void*>(rac_moments_kernel<4>)
                                       : reinterpret_cast<const void*>(rac_moments_kernel<-1>);
    const int64_t mblocks = cfg->tokens < (int64_t)cus * 4 ? cfg->tokens : (int64_t)cus * 4;
    if (hipLaunchKernel(mfn, dim3((unsigned)mblocks), dim3((unsigned)threads), margs, 0, stream) != hipSuccess)
        return RAC_ERR_HIP;
    // 2. merge per (segment, group) into every row's coefficient slot
    void* pargs[] = {&A, &mom};
    const uint64_t pgrid = pblocks < kMaxDispatchItems / (kWave * kPoolWaves) ? pblocks
                                                                              : kMaxDispatchItems / (kWave * kPoolWaves);
    if (hipLaunchKernel(reinterpret_cast<const void*>(rac_pool_kernel), dim3((unsigned)pgrid),
                        dim3(kWave * kPoolWaves), pargs, 0, stream) != hipSuccess)
        return RAC_ERR_HIP;
    // 3. the encode with the pairs given
    A.cf_given = 1;
    A.write_header = 1;
    fill_header(A, cfg, ref == nullptr, true);
    if (use_rows_kernel(A)) return launch(pick_rows(A, cfg->bits), A, stream, kRowsWaves * kWave);
    return launch(pick_encode(A, cfg->bits), A, stream);
}

rac_status rac_reconstruct(const rac_config* cfg, const void* wire, const void* ref,
                           const float* fixed_steps, void* xhat, rac_stream_t stream) {
    return run_decode(cfg, wire, ref, fixed_steps, xhat, stream);
}

rac_status rac_decode(const rac_config* cfg, const void* wire, const void* ref, const float* fixed_steps,
                      void* xhat, rac_stream_t stream) {
    return run_decode(cfg, wire, ref, fixed_steps, xhat, stream);
}

}  // extern "C"

namespace {

uint64_t err_parts(int64_t tokens) { return (uint64_t)((tokens + kErrRows - 1) / kErrRows); }

bool error_args_ok(int64_t tokens, int32_t hidden, uint32_t flags) {
    return tokens >= 0 && tokens <= 0x7FFFFFFFll && hidden >= 8 && hidden % 8 == 0 &&
           (flags & ~uint32_t(RAC_FLAG_XHAT_BF16)) == 0 && (uint64_t)tokens * (uint64_t)hidden < (1ull << 40);
}

// The two launches of the error reduction, with `part` holding err_parts(T)
// partials (3 doubles each).
rac_status run_error(int64_t tokens, int32_t hidden, uint32_t flags, const void* x, const void* xhat,
                     double* stats, double* part, hipStream_t stream) {
    const uint32_t T = (uint32_t)tokens, P = (uint32_t)err_parts(tokens);
    int32_t bf16 = (flags & RAC_FLAG_XHAT_BF16) ? 1 : 0;
    const uint16_t* xp = static_cast<const uint16_t*>(x);
    if (P > 0) {
        uint32_t rows = T;
        void* a[] = {(void*)&xp, (void*)&xhat, (void*)&bf16, (void*)&rows, (void*)&hidden, (void*)&part};
        const uint32_t grid = P < kMaxDispatchItems / kErrThreads ? P : (uint32_t)(kMaxDispatchItems / kErrThreads);
        if (hipLaunchKernel(reinterpret_cast<const void*>(rac_error_kernel), dim3(grid), dim3(kErrThreads), a, 0,
                            stream) != hipSuccess)
            return RAC_ERR_HIP;
    }
    uint32_t np = P;
    void* b[] = {(void*)&part, (void*)&np, (void*)&stats};
    if (hipLaunchKernel(reinterpret_cast<const void*>(rac_error_final_kernel), dim3(1), dim3(kErrThreads), b, 0,
                        stream) != hipSuccess)
        return RAC_ERR_HIP;
    return RAC_OK;
}

rac_status check_error_call(int64_t tokens, int32_t hidden, uint32_t flags, const void* x, const void* xhat,
                            const double* stats) {
    if (!error_args_ok(tokens, hidden, flags) || !stats || (tokens > 0 && (!x || !xhat))) return RAC_ERR_INVALID;
    if (!aligned(x, 16) || !aligned(xhat, 16) || !aligned(stats, 8)) return RAC_ERR_ALIGN;
    return RAC_OK;
}

uint64_t calib_xhat_bytes(const rac_config& c) {
    return (uint64_t)c.tokens * (uint64_t)c.hidden * ((c.flags & RAC_FLAG_XHAT_BF16) ? 2u : 4u);
}

// Workspace of rac_calibrate: x-hat, wire, error partials, per-candidate
// sums, each piece 256-byte aligned.  0 when the candidates are invalid.
struct CalibSpace {
    uint64_t xhat, wire, part, stats, total;
};

bool calib_space(const rac_candidate* c, int32_t n, CalibSpace* out) {
    if (!c || n < 1) return false;
    uint64_t xh = 0, wmax = 0;
    for (int32_t i = 0; i < n; ++i) {
        const rac_config& k = c[i].cfg;
        if (!config_valid(&k) || k.tokens != c[0].cfg.tokens || k.hidden != c[0].cfg.hidden ||
            (k.flags & RAC_FLAG_FIXED_STEP) || k.hidden > kMaxWaves * kChunk)
            return false;
        const uint64_t w = sizes_of(&k).L.total;
        wmax = w > wmax ? w : wmax;
        const uint64_t b = calib_xhat_bytes(k);
        xh = b > xh ? b : xh;
    }
    out->xhat = 0;
    out->wire = up256(xh);
    out->part = out->wire + up256(wmax);
    out->stats = out->part + up256(err_parts(c[0].cfg.tokens) * 24u);
    out->total = out->stats + up256((uint64_t)n * 24u);
    return true;
}

}  // namespace

extern "C" {

size_t rac_recon_error_workspace(int64_t tokens) {
    if (tokens < 0 || tokens > 0x7FFFFFFFll) return 0;
    return (size_t)(err_parts(tokens) * 24u);
}

rac_status rac_recon_error(int64_t tokens, int32_t hidden, uint32_t flags, const void* x, const void* xhat,
                           double* stats, void* workspace, size_t workspace_bytes, rac_stream_t stream) {
    rac_status st = check_error_call(tokens, hidden, flags, x, xhat, stats);
    if (st != RAC_OK) return st;
    if (workspace_bytes < err_parts(tokens) * 24u || (tokens > 0 && !workspace)) return RAC_ERR_CAPACITY;
    if (!aligned(workspace, 8)) return RAC_ERR_ALIGN;
    return run_error(tokens, hidden, flags, x, xhat, stats, static_cast<double*>(workspace), stream);
}

}  // extern "C"

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
double* g_scratch_dev[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
rac_status scratch_address(double** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return RAC_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return RAC_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return RAC_ERR_HIP;
        g_scratch_dev[dev] = static_cast<double*>(p);
    }
    *out = g_scratch_dev[dev];
    return RAC_OK;
}

}  // namespace

extern "C" {

rac_status rac_recon_error_noalloc(int64_t tokens, int32_t hidden, uint32_t flags, const void* x, const void* xhat,
                                   double* stats, rac_stream_t stream) {
    rac_status st = check_error_call(tokens, hidden, flags, x, xhat, stats);
    if (st != RAC_OK) return st;
    if (err_parts(tokens) > kScratchParts) return RAC_ERR_CAPACITY;
    double* part = nullptr;
    if ((st = scratch_address(&part)) != RAC_OK) return st;
    // (every partial the final launch reads is written by the first, so
    // nothing left by an earlier call is read)
    return run_error(tokens, hidden, flags, x, xhat, stats, part, stream);
}

size_t rac_calibrate_workspace(const rac_candidate* candidates, int32_t n) {
    CalibSpace sp;
    return calib_space(candidates, n, &sp) ? (size_t)sp.total : 0;
}

rac_status rac_calibrate(const void* x, const void* ref, rac_candidate* candidates, int32_t n, double target_nmse,
                         void* workspace, size_t workspace_bytes, int32_t* chosen, rac_stream_t stream) {
    CalibSpace sp;
    if (!calib_space(candidates, n, &sp) || !chosen || !x || !(target_nmse >= 0.0)) return RAC_ERR_INVALID;
    if (!workspace || workspace_bytes < sp.total) return RAC_ERR_CAPACITY;
    if (!aligned(workspace, 256) || !aligned(x, 16) || (ref && !aligned(ref, 16))) return RAC_ERR_ALIGN;
    uint8_t* ws = static_cast<uint8_t*>(workspace);
    void* xh = ws + sp.xhat;
    void* wire = ws + sp.wire;
    double* part = reinterpret_cast<double*>(ws + sp.part);
    double* sums = reinterpret_cast<double*>(ws + sp.stats);
    const uint64_t cap = sp.part - sp.wire;
    for (int32_t i = 0; i < n; ++i) {
        const rac_config& c = candidates[i].cfg;
        rac_status st = run_encode(&c, x, ref, nullptr, wire, cap, xh, stream, false, 0, nullptr);
        if (st != RAC_OK) return st;
        st = run_error(c.tokens, c.hidden, c.flags & RAC_FLAG_XHAT_BF16, x, xh, sums + 3 * i, part, stream);
        if (st != RAC_OK) return st;
    }
    // (an offline routine: the results are read back and the stream is
    // synchronized, in chunks of a small host buffer)
    double host[3 * 64];
    for (int32_t i0 = 0; i0 < n; i0 += 64) {
        const int32_t m = n - i0 < 64 ? n - i0 : 64;
        if (hipMemcpyAsync(host, sums + 3 * i0, sizeof(double) * 3u * (size_t)m, hipMemcpyDeviceToHost, stream) !=
                hipSuccess ||
            hipStreamSynchronize(stream) != hipSuccess)
            return RAC_ERR_HIP;
        for (int32_t j = 0; j < m; ++j) {
            rac_candidate& k = candidates[i0 + j];
            k.sq_err = host[3 * j];
            k.sq_x = host[3 * j + 1];
            k.max_abs = host[3 * j + 2];
            k.nmse = k.sq_x > 0.0 ? k.sq_err / k.sq_x : 0.0;
            k.wire_bytes = sizes_of(&k.cfg).L.total;
            k.feasible = k.nmse <= target_nmse ? 1 : 0;
        }
    }
    // fewest wire bytes among the feasible (ties: smaller error, earlier);
    // with none feasible, the smallest error (ties: fewer bytes, earlier)
    int32_t best = -1;
    bool any = false;
    for (int32_t i = 0; i < n; ++i) any = any || candidates[i].feasible;
    for (int32_t i = 0; i < n; ++i) {
        const rac_candidate& k = candidates[i];
        if (any && !k.feasible) continue;
        if (best < 0) {
            best = i;
            continue;
        }
        const rac_candidate& b = candidates[best];
        const bool better = any ? (k.wire_bytes < b.wire_bytes || (k.wire_bytes == b.wire_bytes && k.sq_err < b.sq_err))
                                : (k.sq_err < b.sq_err || (k.sq_err == b.sq_err && k.wire_bytes < b.wire_bytes));
        if (better) best = i;
    }
    *chosen = best;
    return RAC_OK;
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
        case RAC_ERR_NOMEM: return "host memory exhausted";
    }
    return "unknown status";
}

}  // extern "C"
