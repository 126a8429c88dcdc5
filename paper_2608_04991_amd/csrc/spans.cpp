// spans.cpp - host-side selection of the prefill-uplink reference rows
// (subsection "Repeated-Span Retrieval for Prefill Uplinks",
// Eq. prefill-reference-selection).  Produces, for every position of the
// current prompt, the row of the activation store that rac_encode_gather and
// rac_decode_gather read as its reference.
//
// Index: every w-token window of the earlier requests, under a polynomial
// rolling hash (mod 2^64).  Each hash value holds one entry per distinct window
// content (the content is compared token by token, so a hash collision never
// mixes two windows), and each entry keeps its eight most recent occurrences
// in a ring.  Recency is the order of insertion: request order, then position.
//
// Selection: a left-to-right scan over the prompt.  At position i the
// occurrences of the window starting at i are extended forward to their
// longest exact match; the lexicographic maximum of (length, recency) is
// taken and the scan moves past it; without a candidate it moves by one.
#include <stdint.h>

#include <new>
#include <unordered_map>
#include <vector>

#include "rac.h"

namespace {

constexpr int kKeep = 8;                         // occurrences kept per window content
constexpr uint64_t kBase = 0x100000001B3ull;     // odd multiplier of the rolling hash
constexpr int32_t kMaxWindow = 4096;

struct Occ {
    int32_t req;
    int32_t pos;
};

struct Window {
    Occ first;          // an occurrence whose tokens are this entry's content
    Occ ring[kKeep];    // most recent occurrences, oldest overwritten first
    int32_t count;      // occurrences seen (the ring holds min(count, kKeep))
};

uint64_t mix(int32_t t) { return (uint64_t)(uint32_t)t + 1u; }

// hashes of every window of `t` (n - w + 1 of them; none when n < w)
void window_hashes(const int32_t* t, int64_t n, int32_t w, std::vector<uint64_t>& out) {
    out.clear();
    if (n < w) return;
    uint64_t top = 1;  // kBase^(w-1)
    for (int32_t i = 1; i < w; ++i) top *= kBase;
    uint64_t h = 0;
    for (int32_t i = 0; i < w; ++i) h = h * kBase + mix(t[i]);
    out.reserve((size_t)(n - w + 1));
    out.push_back(h);
    for (int64_t j = 1; j + w <= n; ++j) {
        h = (h - mix(t[j - 1]) * top) * kBase + mix(t[j + w - 1]);
        out.push_back(h);
    }
}

}  // namespace

struct rac_span_index {
    int32_t w;
    std::vector<std::vector<int32_t>> reqs;  // token copies of the earlier requests
    std::vector<int64_t> base;               // store row of each request's first token
    std::unordered_map<uint64_t, std::vector<Window>> map;

    bool same(const int32_t* a, const Occ& o) const {
        const int32_t* b = reqs[(size_t)o.req].data() + o.pos;
        for (int32_t i = 0; i < w; ++i)
            if (a[i] != b[i]) return false;
        return true;
    }
};

extern "C" {

rac_span_index* rac_span_index_create(int32_t window) {
    if (window < 1 || window > kMaxWindow) return nullptr;
    rac_span_index* ix = new (std::nothrow) rac_span_index();
    if (ix) ix->w = window;
    return ix;
}

void rac_span_index_destroy(rac_span_index* ix) { delete ix; }

rac_status rac_span_index_add(rac_span_index* ix, const int32_t* tokens, int64_t n, int64_t store_row0) {
    if (!ix || n < 0 || (n > 0 && !tokens) || store_row0 < 0) return RAC_ERR_INVALID;
    if (n > 0x7FFFFFFFll || store_row0 + n > 0x7FFFFFFFll) return RAC_ERR_INVALID;  // int32 store rows
    if (ix->reqs.size() >= 0x7FFFFFFFu) return RAC_ERR_INVALID;
    try {
        ix->reqs.emplace_back(tokens, tokens + n);
        ix->base.push_back(store_row0);
        const int32_t r = (int32_t)(ix->reqs.size() - 1);
        const int32_t* t = ix->reqs.back().data();
        std::vector<uint64_t> hs;
        window_hashes(t, n, ix->w, hs);
        for (size_t j = 0; j < hs.size(); ++j) {
            std::vector<Window>& slot = ix->map[hs[j]];
            Window* win = nullptr;
            for (Window& c : slot)
                if (ix->same(t + j, c.first)) {
                    win = &c;
                    break;
                }
            if (!win) {
                slot.push_back(Window{});
                win = &slot.back();
                win->first = Occ{r, (int32_t)j};
                win->count = 0;
            }
            win->ring[win->count % kKeep] = Occ{r, (int32_t)j};
            ++win->count;
        }
    } catch (const std::bad_alloc&) {
        return RAC_ERR_NOMEM;
    }
    return RAC_OK;
}

rac_status rac_span_select(const rac_span_index* ix, const int32_t* tokens, int64_t n, int32_t* ref_rows,
                           int64_t* covered) {
    if (!ix || n < 0 || (n > 0 && (!tokens || !ref_rows))) return RAC_ERR_INVALID;
    const int32_t w = ix->w;
    int64_t cov = 0;
    try {
        std::vector<uint64_t> hs;
        window_hashes(tokens, n, w, hs);
        int64_t i = 0;
        while (i < n) {
            bool found = false;
            int64_t bl = 0;
            Occ bo{0, 0};
            if (i + w <= n) {
                const auto it = ix->map.find(hs[(size_t)i]);
                if (it != ix->map.end()) {
                    for (const Window& c : it->second) {
                        if (!ix->same(tokens + i, c.first)) continue;
                        const int32_t held = c.count < kKeep ? c.count : kKeep;
                        for (int32_t k = 0; k < held; ++k) {
                            const Occ& o = c.ring[k];
                            const std::vector<int32_t>& tr = ix->reqs[(size_t)o.req];
                            int64_t L = w;
                            while (i + L < n && o.pos + L < (int64_t)tr.size() && tokens[i + L] == tr[(size_t)(o.pos + L)])
                                ++L;
                            // lexicographic (length, request, position)
                            const bool better = !found || L > bl ||
                                                (L == bl && (o.req > bo.req || (o.req == bo.req && o.pos > bo.pos)));
                            if (better) {
                                found = true;
                                bl = L;
                                bo = o;
                            }
                        }
                        break;  // one entry per window content
                    }
                }
            }
            if (!found) {
                ref_rows[i] = -1;
                ++i;
                continue;
            }
            const int64_t row0 = ix->base[(size_t)bo.req] + bo.pos;
            for (int64_t o = 0; o < bl; ++o) ref_rows[i + o] = (int32_t)(row0 + o);
            cov += bl;
            i += bl;
        }
    } catch (const std::bad_alloc&) {
        return RAC_ERR_NOMEM;
    }
    if (covered) *covered = cov;
    return RAC_OK;
}

}  // extern "C"
