// Stage-1 span offsets (Sec. 3.2.1): which audio tokens each fused token
// averages.  The inputs are the ASR segments (a few per second of audio), so
// this is host code; the offsets it returns feed voxzip_fuse_spans.
//
//   1. A segment takes part when its confidence is strictly above the
//      threshold; its times are clipped to [0, t_total_ms].
//   2. Eq. (3): a time tau maps to token floor(L_a * tau / t_total_ms),
//      computed exactly in 64-bit integers; a segment covers the half-open
//      token interval [first, last).
//   3. Segments go in the order (first, last, input order).  A segment that
//      starts inside the tokens already covered starts where they end; an
//      interval left empty, or whose text has no token, is skipped.
//   4. An interval of n tokens whose text has L_t tokens becomes
//      g = min(L_t, n) consecutive groups with boundaries first + floor(j n / g),
//      j = 1..g (sizes differ by at most one).
//   5. Every token outside the intervals is a span of its own, in place.
#include <algorithm>
#include <limits>
#include <vector>

#include "vz_internal.h"

namespace {

struct Interval {
    int64_t first, last;  // token interval [first, last)
    int32_t text;         // text tokens of the segment
    int32_t order;        // position among the kept segments
};

}  // namespace

int32_t vz_build_span_offsets(const int64_t* t_start_ms, const int64_t* t_end_ms, const float* conf,
                              const int32_t* text_len, int32_t n_seg, int64_t t_total_ms, int32_t L_a,
                              float conf_threshold, int32_t* off_out) {
    std::vector<Interval> iv;
    iv.reserve(static_cast<size_t>(n_seg));
    for (int32_t i = 0; i < n_seg; ++i) {
        if (!(conf[i] > conf_threshold)) continue;
        const int64_t t0 = std::max<int64_t>(t_start_ms[i], 0);
        const int64_t t1 = std::min<int64_t>(t_end_ms[i], t_total_ms);
        if (t1 <= t0) continue;
        iv.push_back({int64_t(L_a) * t0 / t_total_ms, int64_t(L_a) * t1 / t_total_ms, text_len[i],
                      static_cast<int32_t>(iv.size())});
    }
    std::sort(iv.begin(), iv.end(), [](const Interval& a, const Interval& b) {
        if (a.first != b.first) return a.first < b.first;
        if (a.last != b.last) return a.last < b.last;
        return a.order < b.order;
    });

    int32_t n = 0;
    off_out[0] = 0;
    int64_t covered = 0;  // tokens [0, covered) belong to emitted spans
    for (const Interval& v : iv) {
        const int64_t a = std::max(v.first, covered), b = v.last;
        if (b <= a || v.text < 1) continue;
        while (covered < a) off_out[++n] = static_cast<int32_t>(++covered);  // background tokens
        const int64_t len = b - a;
        const int64_t groups = std::min<int64_t>(v.text, len);
        for (int64_t j = 1; j <= groups; ++j) off_out[++n] = static_cast<int32_t>(a + j * len / groups);
        covered = b;
    }
    while (covered < L_a) off_out[++n] = static_cast<int32_t>(++covered);
    return n;
}
