// Step table for the fused GELU + requantisation epilogue.
//
// With int8 output, q(y) = clamp(rint(fl(GELU(y) * inv_so)), -127, 127) is a
// step function of the dequantised value y: GELU(erf) is monotone on each
// side of its minimum and rint/clamp keep that, so over a short interval of y
// q changes at most once. The table cuts y into cells (the cell of y is
// clamp(trunc(fma(y, hinv, off)), 0, nc-1), computed the same way on the GPU)
// and stores per cell its code before and after the one change and the exact
// fp32 y where it happens, found by bisection on the fp32 expression itself
// (the same operations, in the same order, as the definition). The kernel
// then needs one compare per output instead of an erf evaluation.
//
// A table whose cells would hold more than one change (output scales below
// about 0.01) is reported as unusable and the kernel evaluates erf instead.
#include <math.h>
#include <string.h>

#include <map>
#include <memory>
#include <mutex>

#include "sl_internal.h"

namespace sl {

static float gelu_f32(float y)
{
    const float t = y * 0.70710678118654752f;
    const float e = erff(t);
    const float h = 0.5f * y;
    const float one_e = 1.0f + e;
    return h * one_e;
}

static int code_of(float y, float inv_so)
{
    const float v = gelu_f32(y) * inv_so;
    float r = rintf(v);
    if (r > 127.0f) r = 127.0f;
    if (r < -127.0f) r = -127.0f;
    return (int)r;
}

// fp32 values ordered as integers (monotone map of the float line)
static int32_t ord(float f)
{
    int32_t i;
    memcpy(&i, &f, 4);
    return i >= 0 ? i : (int32_t)(0x80000000u - (uint32_t)i);
}
static float unord(int32_t o)
{
    const int32_t i = o >= 0 ? o : (int32_t)(0x80000000u - (uint32_t)o);
    float f;
    memcpy(&f, &i, 4);
    return f;
}

static int cell_of(const GeluTable &t, float y)
{
    float c = fmaf(y, t.hinv, t.off);
    const float top = kGeluBase + (float)(t.nc - 1);
    c = c < kGeluBase ? kGeluBase : (c > top ? top : c);
    return (int)(c - kGeluBase);
}

// smallest y in [lo, hi] (as fp32, ordered) with pred(y) true; pred monotone
template <class P>
static float first_true(float lo, float hi, P pred)
{
    int32_t a = ord(lo), b = ord(hi);
    while (a < b) {
        const int32_t mid = a + (int32_t)(((int64_t)b - a) / 2);
        if (pred(unord(mid)))
            b = mid;
        else
            a = mid + 1;
    }
    return unord(a);
}

static std::shared_ptr<GeluTable> build(float inv_so)
{
    auto t = std::make_shared<GeluTable>();
    t->ok = false;
    t->nc = kGeluCells;
    // The cells span only where the code can change: GELU falls from 0 to
    // its minimum (near y = -0.75) and rises after it, so below some kLo <=
    // -1 every code is 0 (the value only shrinks further left) and above some
    // hi every code is 127. Both ends are found by bisection on the
    // expression itself, with a margin; cells of (hi - kLo) / nc then stay
    // narrower than the gap between code changes down to output scales of
    // about 0.01.
    const float far_hi = 130.0f / inv_so + 8.0f;
    if (!isfinite(far_hi) || code_of(far_hi, inv_so) != 127 || code_of(-1e30f, inv_so) != 0) return t;
    float kLo = -1.0f;
    if (code_of(-1.0f, inv_so) != 0)
        kLo = first_true(-1.0e30f, -1.0f, [&](float y) { return code_of(y, inv_so) != 0; }) - 0.5f;
    const float hi = first_true(0.0f, far_hi, [&](float y) { return code_of(y, inv_so) == 127; }) + 0.5f;
    const float h = (hi - kLo) / (float)t->nc;
    t->hinv = 1.0f / h;
    // an integer offset keeps off exact next to kGeluBase
    t->off = kGeluBase + floorf(-kLo * t->hinv);
    if (!(isfinite(t->hinv) && isfinite(t->off))) return t;
    if (code_of(kLo, inv_so) != 0 || code_of(hi, inv_so) != 127) return t;

    float start = -3.0e38f;
    for (int c = 0; c < t->nc; ++c) {
        // [start, end]: the fp32 values whose cell is c
        const float end = c + 1 < t->nc ? unord(ord(first_true(start, 3.0e38f, [&](float y) {
                                             return cell_of(*t, y) > c;
                                         })) - 1)
                                        : 3.0e38f;
        const float a = start < kLo ? kLo : start, b = end > hi ? hi : end;
        const int q0 = code_of(a, inv_so), q1 = code_of(b, inv_so);
        GeluCell &e = t->cell[c];
        e.q_lo = (int8_t)q0;
        e.q_hi = (int8_t)q1;
        e.pad = 0;
        if (q0 == q1) {
            e.thr = INFINITY;
            // a change and a change back inside the cell would be missed
            for (int s = 1; s < 32; ++s) {
                const float y = a + (b - a) * ((float)s / 32.0f);
                if (code_of(y, inv_so) != q0) return t;
            }
        } else {
            const bool up = q1 > q0;
            const float thr = first_true(a, b, [&](float y) {
                const int q = code_of(y, inv_so);
                return up ? q >= q1 : q <= q1;
            });
            e.thr = thr;
            for (int s = 1; s < 32; ++s) {
                const float y = a + (b - a) * ((float)s / 32.0f);
                if (code_of(y, inv_so) != (y >= thr ? q1 : q0)) return t;
            }
        }
        start = unord(ord(end) + 1);
    }
    t->ok = true;
    return t;
}

std::shared_ptr<const GeluTable> gelu_table(float inv_so)
{
    static std::mutex mu;
    static std::map<uint32_t, std::shared_ptr<GeluTable>> cache;
    uint32_t key;
    memcpy(&key, &inv_so, 4);
    {
        std::lock_guard<std::mutex> lk(mu);
        auto it = cache.find(key);
        if (it != cache.end()) return it->second;
    }
    std::shared_ptr<GeluTable> t = build(inv_so);
    std::lock_guard<std::mutex> lk(mu);
    if (cache.size() >= 256) cache.clear();
    cache[key] = t;
    return t;
}

}  // namespace sl
