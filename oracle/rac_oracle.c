/*
 * rac_oracle.c - plain, slow, single-threaded CPU oracle of the RAC aligned
 * residual codec.  TEST INFRASTRUCTURE ONLY (see rac_oracle.h): nothing on the
 * product path links or calls it, and it shares no code with the HIP library.
 *
 * Build: gcc -std=c11 -O2 -ffp-contract=off -fno-fast-math.  Every float
 * operation below is one IEEE-754 binary32 operation rounded to nearest even;
 * contraction into fused multiply-adds is disabled so the text is the
 * arithmetic.
 *
 * Why binary32 and not binary64: every quantity the codec computes feeds a
 * discrete decision (the fp16 wire rounding of alpha/beta, the fp16 scale
 * round-up, the integer codes, the outlier choice).  Both sides must take such
 * decisions in the same precision, which is the kernel's binary32.  The fit
 * is separately pinned against exact rational least squares in the tests.
 *
 * Readings of the paper that are not spelled out there (each one is listed
 * with its justification in the design notes of the repository):
 *   - fit scope is one (alpha, beta) per token row and alignment group;
 *   - the aligned reference alpha*r + beta is rounded once (a fused
 *     multiply-add); with fp16 alpha and bf16 r the product is exact in
 *     binary32 unless it underflows, so this equals the two-step form
 *     everywhere except in that corner, where it fixes one answer;
 *   - sums use the canonical pairwise tree orc_tsum, fit is two-pass centred;
 *   - Round_wire for alpha/beta is fp16 round-to-nearest-even, saturating;
 *   - RoundUp_wire for the scale is "smallest fp16 h with h*Qmax >= max|E^d|";
 *   - the rounding of E/s is round-half-to-even;
 *   - codes are q-bit two's complement, packed LSB-first per token row;
 *   - outliers are the k largest |E| per token row, ties to the lower channel,
 *     emitted in ascending channel order with fp16 values;
 *   - in the per-group outlier mode (the outlier paragraph's own scope) each
 *     quantization group gives up its k_g largest |E|, ties to the lower
 *     channel, listed group by group in ascending in-group offset, the
 *     offsets as u8 and the values as fp16 in two separate arrays;
 *   - q in {2,3} use the same formula as {4,8} (Qmax = 1 and 3).
 */
#include "rac_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define ORC_MAGIC 0x31434152u /* bytes 'R','A','C','1' */
#define ORC_VERSION 2u
#define ORC_HDR 256u
#define ORC_F16_MAX_BITS 0x7BFFu
#define ORC_F16_INF_BITS 0x7C00u
/* The smallest magnitude that round-to-nearest-even fp16 rounds to infinity:
 * the midpoint between 65504 and the next step up, 65536 (a tie, which goes
 * to the even significand, i.e. past the range). */
#define ORC_F16_OVERFLOW 65520.0f

/* ------------------------------------------------------------------------ */
/* Number formats.  Written from the IEEE-754 definitions: an fp16 pattern
 * with exponent field e and fraction m has value m*2^-24 if e == 0, else
 * (1024+m)*2^(e-25).  Rounding is done by locating the two neighbouring
 * representable values and comparing with their exact midpoint.           */

float orc_bf16_to_f32(uint16_t h) {
    uint32_t u = (uint32_t)h << 16; /* bf16 is the top half of binary32 */
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

float orc_f16_to_f32(uint16_t h) {
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 31;
    int m = h & 1023;
    float v;
    if (e == 0)
        v = ldexpf((float)m, -24);
    else if (e == 31)
        v = m ? NAN : INFINITY;
    else
        v = ldexpf((float)(1024 + m), e - 25);
    return sign ? -v : v;
}

uint16_t orc_f16_rne_sat(float f) {
    uint16_t sign = signbit(f) ? 0x8000u : 0u;
    float a = fabsf(f);
    if (a >= 65504.0f) return (uint16_t)(sign | ORC_F16_MAX_BITS);
    /* largest non-negative pattern whose value is <= a; values grow with the
     * pattern over [0, 0x7BFF] */
    uint32_t lo = 0, hi = ORC_F16_MAX_BITS;
    while (lo < hi) {
        uint32_t mid = (lo + hi + 1) / 2;
        if (orc_f16_to_f32((uint16_t)mid) <= a)
            lo = mid;
        else
            hi = mid - 1;
    }
    float below = orc_f16_to_f32((uint16_t)lo);
    float above = orc_f16_to_f32((uint16_t)(lo + 1));
    /* neighbours differ by one fp16 ulp, so their midpoint has at most 13
     * significant bits and is exact in binary32 */
    float half = (below + above) * 0.5f;
    uint32_t p;
    if (a < half)
        p = lo;
    else if (a > half)
        p = lo + 1;
    else
        p = (lo & 1u) ? lo + 1 : lo; /* tie: even fraction */
    return (uint16_t)(sign | p);
}

/* IEEE round-to-nearest-even fp32 -> fp16 with overflow to +-infinity: the
 * rounding the wire's fp16 fields hold, so a saturation is visible there. */
uint16_t orc_f16_rne(float f) {
    if (fabsf(f) >= ORC_F16_OVERFLOW) return (uint16_t)((signbit(f) ? 0x8000u : 0u) | ORC_F16_INF_BITS);
    return orc_f16_rne_sat(f);
}

/* The value a wire fp16 field stands for in the arithmetic of both ends:
 * +-infinity (an overflowed rounding) counts as +-65504. */
float orc_f16_wire(uint16_t h) {
    const float v = orc_f16_to_f32(h);
    const float m = orc_f16_to_f32(ORC_F16_MAX_BITS);
    return v > m ? m : (v < -m ? -m : v);
}

uint16_t orc_f32_to_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    uint32_t sign = u & 0x80000000u;
    uint32_t mag = u & 0x7FFFFFFFu;
    if (mag > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u); /* NaN stays NaN */
    /* the bf16 value below |f| is the truncation, the one above is one unit
     * of the 16-bit pattern higher; compare |f| with their midpoint, which is
     * the truncation with bit 15 set (exact in binary32) */
    uint32_t down = mag & 0xFFFF0000u;
    uint32_t midbits = down | 0x8000u;
    uint32_t p;
    if (mag < midbits)
        p = down >> 16;
    else if (mag > midbits)
        p = (down >> 16) + 1;
    else
        p = ((down >> 16) & 1u) ? (down >> 16) + 1 : (down >> 16);
    return (uint16_t)((sign >> 16) | p);
}

uint16_t orc_scale_roundup(float m, int32_t qmax) {
    /* value(h)*qmax is exact in binary32 (11-bit by 7-bit significands), so
     * the predicate is an exact comparison and is monotone in h */
    const float q = (float)qmax;
    /* no finite fp16 covers m: the upward rounding goes past the range */
    if (orc_f16_to_f32(ORC_F16_MAX_BITS) * q < m) return ORC_F16_INF_BITS;
    uint32_t lo = 1, hi = ORC_F16_MAX_BITS;
    while (lo < hi) {
        uint32_t mid = (lo + hi) / 2;
        if (orc_f16_to_f32((uint16_t)mid) * q >= m)
            hi = mid;
        else
            lo = mid + 1;
    }
    return (uint16_t)lo;
}

uint16_t orc_step_roundup(float step) {
    if (orc_f16_to_f32(ORC_F16_MAX_BITS) < step) return ORC_F16_MAX_BITS;
    uint32_t lo = 1, hi = ORC_F16_MAX_BITS;
    while (lo < hi) {
        uint32_t mid = (lo + hi) / 2;
        if (orc_f16_to_f32((uint16_t)mid) >= step)
            hi = mid;
        else
            lo = mid + 1;
    }
    return (uint16_t)lo;
}

/* ------------------------------------------------------------------------ */
/* Canonical sum: a perfect pairwise tree over channel order.                */
float orc_tsum(const float* v, int32_t n) {
    if (n == 1) return v[0];
    int32_t h = n / 2;
    return orc_tsum(v, h) + orc_tsum(v + h, n - h);
}

/* Eq. affine-fit: least squares of x ~ alpha*r + beta over one group, solved
 * in closed form with centred moments: alpha* = C_rx / C_rr and
 * beta* = mean(x) - alpha* mean(r).  A reference group with zero variance
 * gives alpha* = 0, beta* = mean(x), as the paper prescribes.  beta* uses the
 * unrounded alpha*: the paper rounds the solved pair to the wire format. */
void orc_fit_group(const float* r, const float* x, int32_t g, float* alpha_star,
                   float* beta_star) {
    float* uu = (float*)malloc(sizeof(float) * (size_t)g);
    float* uv = (float*)malloc(sizeof(float) * (size_t)g);
    const float mr = orc_tsum(r, g) / (float)g;
    const float mx = orc_tsum(x, g) / (float)g;
    for (int32_t c = 0; c < g; ++c) {
        const float u = r[c] - mr;
        const float v = x[c] - mx;
        uu[c] = u * u;
        uv[c] = u * v;
    }
    const float crr = orc_tsum(uu, g);
    const float crx = orc_tsum(uv, g);
    free(uu);
    free(uv);
    if (crr == 0.0f) {
        *alpha_star = 0.0f;
        *beta_star = mx;
    } else {
        const float a = crx / crr;
        *alpha_star = a;
        *beta_star = mx - a * mr;
    }
}

/* ------------------------------------------------------------------------ */
/* Outlier choice: sort every channel by (larger |e| first, lower channel
 * first) and keep the first k, then list them in ascending channel order.   */
typedef struct {
    float mag;
    int32_t idx;
} orc_cand;

static int orc_cmp_rank(const void* pa, const void* pb) {
    const orc_cand* a = (const orc_cand*)pa;
    const orc_cand* b = (const orc_cand*)pb;
    if (a->mag > b->mag) return -1;
    if (a->mag < b->mag) return 1;
    return (a->idx < b->idx) ? -1 : (a->idx > b->idx);
}

static int orc_cmp_u16(const void* pa, const void* pb) {
    uint16_t a = *(const uint16_t*)pa, b = *(const uint16_t*)pb;
    return (a > b) - (a < b);
}

void orc_topk_row(const float* e, int32_t d, int32_t k, uint16_t* idx) {
    orc_cand* all = (orc_cand*)malloc(sizeof(orc_cand) * (size_t)d);
    for (int32_t c = 0; c < d; ++c) {
        all[c].mag = fabsf(e[c]);
        all[c].idx = c;
    }
    qsort(all, (size_t)d, sizeof(orc_cand), orc_cmp_rank);
    for (int32_t i = 0; i < k; ++i) idx[i] = (uint16_t)all[i].idx;
    free(all);
    qsort(idx, (size_t)k, sizeof(uint16_t), orc_cmp_u16);
}

/* ------------------------------------------------------------------------ */
/* Wire layout: a 256-byte header, then coefficient, scale, code and outlier
 * sections, each starting at a 256-byte boundary; all padding is zero.      */

static int is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

static int orc_valid(const orc_config* c) {
    if (!c) return 0;
    if (c->tokens < 0 || c->tokens > 0xFFFFFFFFll) return 0;
    if (c->hidden < 8 || c->hidden > 65535 || (c->hidden % 8) != 0) return 0;
    if (!is_pow2(c->group_align) || c->group_align < 8 || c->group_align > c->hidden ||
        c->hidden % c->group_align != 0)
        return 0;
    if (!is_pow2(c->group_quant) || c->group_quant < 8 || c->group_quant > c->hidden ||
        c->hidden % c->group_quant != 0)
        return 0;
    if (c->bits != 2 && c->bits != 3 && c->bits != 4 && c->bits != 8) return 0;
    if (c->flags & ~(uint32_t)(ORC_FLAG_FIXED_STEP | ORC_FLAG_XHAT_BF16 | ORC_FLAG_GROUP_OUTLIERS))
        return 0;
    if (c->flags & ORC_FLAG_GROUP_OUTLIERS) {
        /* u8 in-group offsets, and at most a quarter of a group set aside */
        if (c->group_quant > 256) return 0;
        if (c->outlier_k < 1 || c->outlier_k > 16 || c->outlier_k > c->group_quant / 4) return 0;
    } else if (c->outlier_k < 0 || c->outlier_k > 64 || c->outlier_k > c->hidden) {
        return 0;
    }
    return 1;
}

static uint64_t up256(uint64_t v) { return (v + 255u) & ~(uint64_t)255u; }


int orc_layout_of(const orc_config* cfg, orc_layout* out) {
    if (!orc_valid(cfg) || !out) return ORC_ERR_INVALID;
    const uint64_t T = (uint64_t)cfg->tokens, d = (uint64_t)cfg->hidden;
    const uint64_t coef = T * (d / (uint64_t)cfg->group_align) * 4u;
    const uint64_t scale =
        (cfg->flags & ORC_FLAG_FIXED_STEP) ? 0u : T * (d / (uint64_t)cfg->group_quant) * 2u;
    const uint64_t codes = T * d * (uint64_t)cfg->bits / 8u;
    out->off_coef = ORC_HDR;
    out->off_scale = up256(out->off_coef + coef);
    out->off_codes = up256(out->off_scale + scale);
    out->off_outl = up256(out->off_codes + codes);
    if (cfg->flags & ORC_FLAG_GROUP_OUTLIERS) {
        /* fp16 values [T][d/g_q][k_g], then u8 offsets [T][d/g_q][k_g] */
        const uint64_t n = T * (d / (uint64_t)cfg->group_quant) * (uint64_t)cfg->outlier_k;
        out->off_ooff = up256(out->off_outl + 2u * n);
        out->total = up256(out->off_ooff + n);
    } else {
        out->off_ooff = 0;
        out->total = up256(out->off_outl + T * (uint64_t)cfg->outlier_k * 4u);
    }
    return ORC_OK;
}

static void put16(uint8_t* p, uint16_t v) {
    p[0] = (uint8_t)(v & 0xFF);
    p[1] = (uint8_t)(v >> 8);
}
static void put32(uint8_t* p, uint32_t v) {
    for (int i = 0; i < 4; ++i) p[i] = (uint8_t)(v >> (8 * i));
}
static void put64(uint8_t* p, uint64_t v) {
    for (int i = 0; i < 8; ++i) p[i] = (uint8_t)(v >> (8 * i));
}
static uint16_t get16(const uint8_t* p) { return (uint16_t)(p[0] | (p[1] << 8)); }
static uint32_t get32(const uint8_t* p) {
    return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) | ((uint32_t)p[3] << 24);
}
static uint64_t get64(const uint8_t* p) {
    uint64_t v = 0;
    for (int i = 7; i >= 0; --i) v = (v << 8) | p[i];
    return v;
}

static uint16_t orc_wire_flags(const orc_config* cfg, int zero_ref) {
    uint16_t f = 0;
    const int grouped = (cfg->flags & ORC_FLAG_GROUP_OUTLIERS) != 0;
    if (cfg->outlier_k > 0 && !grouped) f |= 1u;
    if (cfg->flags & ORC_FLAG_FIXED_STEP) f |= 2u;
    if (zero_ref) f |= 4u;
    if (grouped) f |= 8u;
    return f;
}

static void orc_write_header(const orc_config* cfg, const orc_layout* L, int zero_ref,
                             uint8_t* w) {
    put32(w + 0, ORC_MAGIC);
    put16(w + 4, ORC_VERSION);
    put16(w + 6, orc_wire_flags(cfg, zero_ref));
    put32(w + 8, (uint32_t)cfg->tokens);
    put32(w + 12, (uint32_t)cfg->hidden);
    put32(w + 16, (uint32_t)cfg->group_align);
    put32(w + 20, (uint32_t)cfg->group_quant);
    w[24] = (uint8_t)cfg->bits;
    w[25] = 1; /* coefficients: fp16 (alpha, beta) pairs */
    w[26] = (cfg->flags & ORC_FLAG_FIXED_STEP) ? 0 : 1; /* scales: fp16 or absent */
    /* outliers: 1 = u32 (u16 channel | fp16 value) per token, 2 = fp16 values
     * and u8 in-group offsets per quantization group */
    w[27] = (cfg->flags & ORC_FLAG_GROUP_OUTLIERS) ? 2 : (cfg->outlier_k > 0 ? 1 : 0);
    put16(w + 28, (uint16_t)cfg->outlier_k);
    put64(w + 32, L->off_coef);
    put64(w + 40, L->off_scale);
    put64(w + 48, L->off_codes);
    put64(w + 56, L->off_outl);
    put64(w + 64, L->total);
    put64(w + 72, L->off_ooff);
}

/* q-bit two's complement code of channel c goes to bits [c*q, c*q+q) of the
 * row's little-endian bit string (so INT4 keeps even channels in the low
 * nibble, two values per byte). */
static void orc_put_code(uint8_t* row, int32_t c, int32_t bits, int32_t q) {
    const uint32_t u = (uint32_t)q & ((1u << bits) - 1u);
    for (int32_t b = 0; b < bits; ++b) {
        if ((u >> b) & 1u) {
            const int64_t pos = (int64_t)c * bits + b;
            row[pos / 8] |= (uint8_t)(1u << (pos % 8));
        }
    }
}

static int32_t orc_get_code(const uint8_t* row, int32_t c, int32_t bits) {
    uint32_t u = 0;
    for (int32_t b = 0; b < bits; ++b) {
        const int64_t pos = (int64_t)c * bits + b;
        if ((row[pos / 8] >> (pos % 8)) & 1u) u |= 1u << b;
    }
    if (u & (1u << (bits - 1))) return (int32_t)u - (1 << bits); /* sign */
    return (int32_t)u;
}

static void orc_store_xhat(const orc_config* cfg, void* xhat, int64_t i, float v) {
    if (cfg->flags & ORC_FLAG_XHAT_BF16)
        ((uint16_t*)xhat)[i] = orc_f32_to_bf16(v);
    else
        ((float*)xhat)[i] = v;
}

/* ------------------------------------------------------------------------ */
/* pooled: NULL for the per-token fit, else [T][d/g_a][2] unrounded (alpha*,
 * beta*) of each row's segment; pooled_flag marks the header. */
static int orc_encode_impl(const orc_config* cfg, const uint16_t* x, const uint16_t* ref,
                           const float* steps, uint8_t* wire, size_t wire_cap, void* xhat,
                           const float* pooled) {
    orc_layout L;
    if (orc_layout_of(cfg, &L) != ORC_OK || !wire) return ORC_ERR_INVALID;
    if ((cfg->flags & ORC_FLAG_FIXED_STEP) && !steps) return ORC_ERR_INVALID;
    if (cfg->tokens > 0 && !x) return ORC_ERR_INVALID;
    if (wire_cap < L.total) return ORC_ERR_CAPACITY;

    const int64_t T = cfg->tokens;
    const int32_t d = cfg->hidden, ga = cfg->group_align, gq = cfg->group_quant;
    const int32_t bits = cfg->bits, k = cfg->outlier_k;
    const int32_t qmax = (1 << (bits - 1)) - 1; /* Eq. residual-quantization */
    const int fixed = (cfg->flags & ORC_FLAG_FIXED_STEP) != 0;
    const int grouped = (cfg->flags & ORC_FLAG_GROUP_OUTLIERS) != 0;

    for (int64_t i = 0; i < T * d; ++i) {
        if (!isfinite(orc_bf16_to_f32(x[i]))) return ORC_ERR_NONFINITE;
        if (ref && !isfinite(orc_bf16_to_f32(ref[i]))) return ORC_ERR_NONFINITE;
    }

    memset(wire, 0, L.total);
    orc_write_header(cfg, &L, ref == NULL, wire);
    if (pooled) put16(wire + 6, (uint16_t)(get16(wire + 6) | 16u)); /* coefficients pooled over segments */

    float* r = (float*)malloc(sizeof(float) * (size_t)d);
    float* xv = (float*)malloc(sizeof(float) * (size_t)d);
    float* rt = (float*)malloc(sizeof(float) * (size_t)d);
    float* e = (float*)malloc(sizeof(float) * (size_t)d);
    float* ed = (float*)malloc(sizeof(float) * (size_t)d);
    uint16_t* oval = (uint16_t*)calloc((size_t)d, sizeof(uint16_t));
    uint8_t* is_out = (uint8_t*)calloc((size_t)d, 1);
    uint16_t sel[64];

    for (int64_t t = 0; t < T; ++t) {
        /* step 1: widen the row (exact) */
        for (int32_t c = 0; c < d; ++c) {
            xv[c] = orc_bf16_to_f32(x[t * d + c]);
            r[c] = ref ? orc_bf16_to_f32(ref[t * d + c]) : 0.0f;
        }
        /* step 2: grouped affine alignment (Eq. affine-fit), serialized to
         * fp16, then the aligned reference and residual (Eq. aligned-residual)
         * formed with the serialized coefficients */
        uint8_t* coef = wire + L.off_coef + (uint64_t)t * (uint64_t)(d / ga) * 4u;
        for (int32_t j = 0; j < d / ga; ++j) {
            float as, bs;
            if (pooled) {
                as = pooled[((uint64_t)t * (uint64_t)(d / ga) + (uint64_t)j) * 2u];
                bs = pooled[((uint64_t)t * (uint64_t)(d / ga) + (uint64_t)j) * 2u + 1u];
            } else {
                orc_fit_group(r + j * ga, xv + j * ga, ga, &as, &bs);
            }
            /* Round_wire: fp16 (+-infinity past the range, read as +-65504) */
            const uint16_t ah = orc_f16_rne(as), bh = orc_f16_rne(bs);
            put16(coef + 4 * j, ah);
            put16(coef + 4 * j + 2, bh);
            const float a = orc_f16_wire(ah), b0 = orc_f16_wire(bh);
            for (int32_t c = j * ga; c < (j + 1) * ga; ++c) {
                rt[c] = fmaf(a, r[c], b0);
                e[c] = xv[c] - rt[c];
            }
        }
        /* step 3: dense / outlier split (mask M over the k largest |E|) */
        memset(is_out, 0, (size_t)d);
        for (int32_t c = 0; c < d; ++c) ed[c] = e[c];
        if (grouped) {
            /* the k_g largest |E| of every quantization group (the outlier
             * paragraph's mask M_j per fixed group) */
            const uint64_t n = (uint64_t)(d / gq) * (uint64_t)k;
            uint8_t* vrow = wire + L.off_outl + (uint64_t)t * n * 2u;
            uint8_t* orow = wire + L.off_ooff + (uint64_t)t * n;
            for (int32_t g = 0; g < d / gq; ++g) {
                orc_topk_row(e + g * gq, gq, k, sel); /* ascending in-group offsets */
                for (int32_t i = 0; i < k; ++i) {
                    const int32_t c = g * gq + sel[i];
                    oval[c] = orc_f16_rne(e[c]);
                    is_out[c] = 1;
                    ed[c] = 0.0f;
                    put16(vrow + 2 * ((uint64_t)g * k + i), oval[c]);
                    orow[(uint64_t)g * k + i] = (uint8_t)sel[i];
                }
            }
        } else if (k > 0) {
            orc_topk_row(e, d, k, sel);
            uint8_t* ol = wire + L.off_outl + (uint64_t)t * (uint64_t)k * 4u;
            for (int32_t i = 0; i < k; ++i) {
                const int32_t c = sel[i];
                oval[c] = orc_f16_rne(e[c]); /* O-hat = Round_FP16(O) */
                is_out[c] = 1;
                ed[c] = 0.0f;
                put32(ol + 4 * i, (uint32_t)c | ((uint32_t)oval[c] << 16));
            }
        }
        /* steps 4-6: per quantization group scale, codes, packing, and the
         * sender-side reconstruction (Eq. residual-reconstruction) */
        uint8_t* crow = wire + L.off_codes + (uint64_t)t * (uint64_t)d * (uint64_t)bits / 8u;
        uint8_t* srow = wire + L.off_scale + (uint64_t)t * (uint64_t)(d / gq) * 2u;
        for (int32_t g = 0; g < d / gq; ++g) {
            uint16_t sh;
            if (fixed) {
                sh = orc_step_roundup(steps[g]);
            } else {
                float m = 0.0f;
                for (int32_t c = g * gq; c < (g + 1) * gq; ++c)
                    if (fabsf(ed[c]) > m) m = fabsf(ed[c]);
                sh = (m == 0.0f) ? 0u : orc_scale_roundup(m, qmax); /* 0 = zero group */
                put16(srow + 2 * g, sh);
            }
            const float s = orc_f16_wire(sh);
            for (int32_t c = g * gq; c < (g + 1) * gq; ++c) {
                int32_t q = 0;
                if (sh != 0u) { /* a zero group skips the division */
                    const float tq = ed[c] / s;
                    float rq = rintf(tq); /* round half to even */
                    if (rq > (float)qmax) rq = (float)qmax;
                    if (rq < (float)-qmax) rq = (float)-qmax;
                    q = (int32_t)rq;
                }
                orc_put_code(crow, c, bits, q);
                if (xhat) {
                    const float eh = is_out[c] ? orc_f16_wire(oval[c]) : (float)q * s;
                    orc_store_xhat(cfg, xhat, t * d + c, rt[c] + eh);
                }
            }
        }
    }
    free(r);
    free(xv);
    free(rt);
    free(e);
    free(ed);
    free(oval);
    free(is_out);
    return ORC_OK;
}

int orc_encode(const orc_config* cfg, const uint16_t* x, const uint16_t* ref,
               const float* steps, uint8_t* wire, size_t wire_cap, void* xhat) {
    return orc_encode_impl(cfg, x, ref, steps, wire, wire_cap, xhat, NULL);
}

/* ------------------------------------------------------------------------ */
/* Fit pooled over segments of rows (the affine-fit equation over all fitting
 * positions of a segment, for example one retrieved span).  Each (row, group)
 * gives its two-pass centred moments exactly as the per-token fit does; the
 * rows of a segment are combined by the pairwise merge of centred moments
 * (Chan, Golub and LeVeque) over the binary-decomposition tree: a range of n
 * rows splits into its first p rows, p the largest power of two below n, and
 * the rest.  A one-row segment is the per-token fit, bit for bit. */

void orc_moments_row(const float* r, const float* x, int32_t g, orc_moments* m) {
    float* uu = (float*)malloc(sizeof(float) * (size_t)g);
    float* uv = (float*)malloc(sizeof(float) * (size_t)g);
    m->n = (float)g;
    m->mr = orc_tsum(r, g) / (float)g;
    m->mx = orc_tsum(x, g) / (float)g;
    for (int32_t c = 0; c < g; ++c) {
        const float u = r[c] - m->mr;
        const float v = x[c] - m->mx;
        uu[c] = u * u;
        uv[c] = u * v;
    }
    m->crr = orc_tsum(uu, g);
    m->crx = orc_tsum(uv, g);
    free(uu);
    free(uv);
}

void orc_moments_merge(const orc_moments* a, const orc_moments* b, orc_moments* o) {
    const float n = a->n + b->n;
    const float dr = b->mr - a->mr;
    const float dx = b->mx - a->mx;
    const float fb = b->n / n;
    const float w = (a->n * b->n) / n;
    orc_moments m;
    m.n = n;
    m.mr = a->mr + dr * fb;
    m.mx = a->mx + dx * fb;
    m.crr = (a->crr + b->crr) + (dr * dr) * w;
    m.crx = (a->crx + b->crx) + (dr * dx) * w;
    *o = m;
}

static void orc_pool_range(const orc_moments* rows, int64_t n, orc_moments* out) {
    if (n == 1) {
        *out = rows[0];
        return;
    }
    int64_t p = 1;
    while (p * 2 < n) p *= 2;
    orc_moments a, b;
    orc_pool_range(rows, p, &a);
    orc_pool_range(rows + p, n - p, &b);
    orc_moments_merge(&a, &b, out);
}

void orc_moments_pool(const orc_moments* rows, int64_t n, orc_moments* out) { orc_pool_range(rows, n, out); }

int orc_encode_pooled(const orc_config* cfg, const uint16_t* x, const uint16_t* ref, int64_t segments,
                      const int32_t* seg_start, const float* steps, uint8_t* wire, size_t wire_cap,
                      void* xhat) {
    orc_layout L;
    if (orc_layout_of(cfg, &L) != ORC_OK || !seg_start) return ORC_ERR_INVALID;
    const int64_t T = cfg->tokens;
    const int32_t d = cfg->hidden, ga = cfg->group_align, G = d / ga;
    if (segments < 1 || segments > T || seg_start[0] != 0 || seg_start[segments] != T) return ORC_ERR_INVALID;
    for (int64_t s = 0; s < segments; ++s)
        if (seg_start[s + 1] <= seg_start[s]) return ORC_ERR_INVALID;
    if (!x) return ORC_ERR_INVALID;
    for (int64_t i = 0; i < T * d; ++i) {
        if (!isfinite(orc_bf16_to_f32(x[i]))) return ORC_ERR_NONFINITE;
        if (ref && !isfinite(orc_bf16_to_f32(ref[i]))) return ORC_ERR_NONFINITE;
    }
    orc_moments* mom = (orc_moments*)malloc(sizeof(orc_moments) * (size_t)(T * G));
    float* pooled = (float*)malloc(sizeof(float) * 2u * (size_t)(T * G));
    float* r = (float*)malloc(sizeof(float) * (size_t)ga);
    float* xv = (float*)malloc(sizeof(float) * (size_t)ga);
    orc_moments* seg = (orc_moments*)malloc(sizeof(orc_moments) * (size_t)T);
    for (int64_t t = 0; t < T; ++t)
        for (int32_t j = 0; j < G; ++j) {
            for (int32_t c = 0; c < ga; ++c) {
                xv[c] = orc_bf16_to_f32(x[t * d + j * ga + c]);
                r[c] = ref ? orc_bf16_to_f32(ref[t * d + j * ga + c]) : 0.0f;
            }
            orc_moments_row(r, xv, ga, &mom[t * G + j]);
        }
    for (int64_t s = 0; s < segments; ++s) {
        const int64_t lo = seg_start[s], n = seg_start[s + 1] - seg_start[s];
        for (int32_t j = 0; j < G; ++j) {
            for (int64_t i = 0; i < n; ++i) seg[i] = mom[(lo + i) * G + j];
            orc_moments m;
            orc_moments_pool(seg, n, &m);
            float a, b;
            if (m.crr == 0.0f) { /* zero-variance reference: (0, mean x) */
                a = 0.0f;
                b = m.mx;
            } else {
                a = m.crx / m.crr;
                b = m.mx - a * m.mr;
            }
            for (int64_t i = 0; i < n; ++i) {
                pooled[((lo + i) * G + j) * 2] = a;
                pooled[((lo + i) * G + j) * 2 + 1] = b;
            }
        }
    }
    const int rc = orc_encode_impl(cfg, x, ref, steps, wire, wire_cap, xhat, pooled);
    free(mom);
    free(pooled);
    free(r);
    free(xv);
    free(seg);
    return rc;
}

int orc_decode(const orc_config* cfg, const uint8_t* wire, const uint16_t* ref,
               const float* steps, void* xhat) {
    orc_layout L;
    if (orc_layout_of(cfg, &L) != ORC_OK || !wire) return ORC_ERR_INVALID;
    if ((cfg->flags & ORC_FLAG_FIXED_STEP) && !steps) return ORC_ERR_INVALID;
    if (cfg->tokens > 0 && !xhat) return ORC_ERR_INVALID;
    /* the header must describe exactly this configuration */
    if (get32(wire + 0) != ORC_MAGIC || get16(wire + 4) != ORC_VERSION) return ORC_ERR_FORMAT;
    const uint16_t wf = get16(wire + 6);
    if ((wf & 11u) != (orc_wire_flags(cfg, 0) & 11u)) return ORC_ERR_FORMAT;
    if (get32(wire + 8) != (uint32_t)cfg->tokens || get32(wire + 12) != (uint32_t)cfg->hidden ||
        get32(wire + 16) != (uint32_t)cfg->group_align ||
        get32(wire + 20) != (uint32_t)cfg->group_quant || wire[24] != (uint8_t)cfg->bits ||
        get16(wire + 28) != (uint16_t)cfg->outlier_k || get64(wire + 32) != L.off_coef ||
        get64(wire + 40) != L.off_scale || get64(wire + 48) != L.off_codes ||
        get64(wire + 56) != L.off_outl || get64(wire + 64) != L.total ||
        get64(wire + 72) != L.off_ooff)
        return ORC_ERR_FORMAT;

    const int64_t T = cfg->tokens;
    const int32_t d = cfg->hidden, ga = cfg->group_align, gq = cfg->group_quant;
    const int32_t bits = cfg->bits, k = cfg->outlier_k;
    const int fixed = (cfg->flags & ORC_FLAG_FIXED_STEP) != 0;
    const int grouped = (cfg->flags & ORC_FLAG_GROUP_OUTLIERS) != 0;
    float* eh = (float*)malloc(sizeof(float) * (size_t)d);
    for (int64_t t = 0; t < T; ++t) {
        const uint8_t* crow = wire + L.off_codes + (uint64_t)t * (uint64_t)d * (uint64_t)bits / 8u;
        const uint8_t* srow = wire + L.off_scale + (uint64_t)t * (uint64_t)(d / gq) * 2u;
        const uint8_t* coef = wire + L.off_coef + (uint64_t)t * (uint64_t)(d / ga) * 4u;
        /* dequantized dense residual DQ(q; s) */
        for (int32_t g = 0; g < d / gq; ++g) {
            const uint16_t sh = fixed ? orc_step_roundup(steps[g]) : get16(srow + 2 * g);
            const float s = orc_f16_wire(sh);
            for (int32_t c = g * gq; c < (g + 1) * gq; ++c)
                eh[c] = (float)orc_get_code(crow, c, bits) * s;
        }
        /* restore the outliers at their channels */
        if (grouped) {
            const uint64_t n = (uint64_t)(d / gq) * (uint64_t)k;
            const uint8_t* vrow = wire + L.off_outl + (uint64_t)t * n * 2u;
            const uint8_t* orow = wire + L.off_ooff + (uint64_t)t * n;
            for (int32_t g = 0; g < d / gq; ++g) {
                for (int32_t i = 0; i < k; ++i) {
                    const uint32_t o = orow[(uint64_t)g * k + i];
                    if (o >= (uint32_t)gq) {
                        free(eh);
                        return ORC_ERR_FORMAT;
                    }
                    eh[g * gq + (int32_t)o] = orc_f16_wire(get16(vrow + 2 * ((uint64_t)g * k + i)));
                }
            }
        } else if (k > 0) {
            const uint8_t* ol = wire + L.off_outl + (uint64_t)t * (uint64_t)k * 4u;
            for (int32_t i = 0; i < k; ++i) {
                const uint32_t w = get32(ol + 4 * i);
                const uint32_t c = w & 0xFFFFu;
                if (c >= (uint32_t)d) {
                    free(eh);
                    return ORC_ERR_FORMAT;
                }
                eh[c] = orc_f16_wire((uint16_t)(w >> 16));
            }
        }
        /* H-hat = R-tilde + E-hat with R-tilde from the serialized alignment */
        for (int32_t j = 0; j < d / ga; ++j) {
            const float a = orc_f16_wire(get16(coef + 4 * j));
            const float b0 = orc_f16_wire(get16(coef + 4 * j + 2));
            for (int32_t c = j * ga; c < (j + 1) * ga; ++c) {
                const float r = ref ? orc_bf16_to_f32(ref[t * d + c]) : 0.0f;
                const float rt = fmaf(a, r, b0);
                orc_store_xhat(cfg, xhat, t * d + c, rt + eh[c]);
            }
        }
    }
    free(eh);
    return ORC_OK;
}
