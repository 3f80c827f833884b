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
//
// GELU falls to its minimum near y = -0.7518 and rises after it, so a code
// can dip and come back inside one interval of y. A cell boundary is placed at
// that minimum: every cell then lies on one side of it, where the code is
// monotone in y, and "at most one change" follows from the codes at the
// cell's two ends. The two cells that meet at the minimum, where the fp32
// expression is flattest, are also checked value by value over every fp32 y
// they hold.
#include <math.h>
#include <string.h>

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

// The minimum of GELU(y) = y Phi(y): Phi(y) + y phi(y) = 0.
constexpr double kGeluMinY = -0.751791524693564457;

// Every fp32 value of [a, b], in order. The codes must change at most once,
// except that the fp32 expression is itself not monotone within a few ulps
// of a rounding boundary where GELU is flat: changes that all fall inside a
// band of at most kNoiseUlps values count as one, and the threshold is put
// where it disagrees with the fewest values of the band (a code differing by
// one, only where the fp32 evaluation itself flips back and forth).
constexpr int kNoiseUlps = 256;

static bool exact_cell(float a, float b, float inv_so, GeluCell *e)
{
    const int q0 = code_of(a, inv_so);
    int q_end = q0, other = q0;
    int32_t first = 0, last = 0;
    bool any = false;
    for (int32_t o = ord(a); o <= ord(b); ++o) {
        const int q = code_of(unord(o), inv_so);
        if (q != q_end) {
            if (!any) first = o;
            last = o;
            any = true;
            if (q != q0) {
                if (other != q0 && q != other) return false;  // a third code
                other = q;
            }
            q_end = q;
        }
    }
    e->q_lo = (int8_t)q0;
    e->q_hi = (int8_t)q_end;
    e->pad = 0;
    e->thr = INFINITY;
    if (!any) return true;
    if ((int64_t)last - first > kNoiseUlps) {
        // changes spread wider than noise: allowed only as one clean change
        int changes = 0, prev = q0;
        for (int32_t o = first; o <= last; ++o) {
            const int q = code_of(unord(o), inv_so);
            if (q != prev) ++changes, prev = q;
        }
        if (changes != 1) return false;
        e->thr = unord(first);
        return true;
    }
    // best single threshold inside the band [first - 1, last]: q0 below it and
    // q_end from it on (no threshold at all when q_end == q0)
    if (q_end == q0) {
        e->thr = INFINITY;
        return true;
    }
    int best_miss = 1 << 30;
    int32_t best = first;
    for (int32_t t = first; t <= last; ++t) {
        int miss = 0;
        for (int32_t o = first - 1; o <= last; ++o) {
            const int q = code_of(unord(o), inv_so);
            miss += o < t ? q != q0 : q != q_end;
        }
        if (miss < best_miss) best_miss = miss, best = t;
    }
    e->thr = unord(best);
    return true;
}

static double gelu_exact(double y) { return 0.5 * y * (1.0 + erf(y * 0.70710678118654752440)); }

// true (and the cell set to that code) when GELU over [a, b], scaled by
// inv_so, lies inside one rounding interval (k - 1/2, k + 1/2) with a margin:
// GELU is unimodal, so its maximum over [a, b] is at an end and its minimum
// at an end or at GELU's minimum
static bool one_code_cell(float a, float b, float inv_so, GeluCell *e)
{
    const double ga = gelu_exact(a), gb = gelu_exact(b);
    double lo = ga < gb ? ga : gb;
    const double hi = ga < gb ? gb : ga;
    if ((double)a <= kGeluMinY && kGeluMinY <= (double)b) lo = gelu_exact(kGeluMinY);
    const double vlo = lo * inv_so, vhi = hi * inv_so;
    const double margin = 1e-4 + 1e-5 * (fabs(vlo) > fabs(vhi) ? fabs(vlo) : fabs(vhi));
    const double k0 = floor(vlo - margin + 0.5), k1 = floor(vhi + margin + 0.5);
    if (k0 != k1) return false;
    const int q = code_of(a, inv_so);
    const double kc = k0 > 127.0 ? 127.0 : (k0 < -127.0 ? -127.0 : k0);
    if ((double)q != kc) return false;
    e->q_lo = e->q_hi = (int8_t)q;
    e->thr = INFINITY;
    e->pad = 0;
    return true;
}

static void build(float inv_so, GeluTable *t)
{
    t->ok = false;
    t->nc = kGeluCells;
    // The cells span only where the code can change: GELU falls from 0 to
    // its minimum and rises after it, so below some kLo <= -1 every code is 0
    // (the value only shrinks further left) and above some hi every code is
    // 127. Both ends are found by bisection on the expression itself, with a
    // margin; cells of (hi - kLo) / nc then stay narrower than the gap
    // between code changes down to output scales of about 0.01.
    const float far_hi = 130.0f / inv_so + 8.0f;
    if (!isfinite(far_hi) || code_of(far_hi, inv_so) != 127 || code_of(-1e30f, inv_so) != 0) return;
    float kLo = -1.0f;
    if (code_of(-1.0f, inv_so) != 0)
        kLo = first_true(-1.0e30f, -1.0f, [&](float y) { return code_of(y, inv_so) != 0; }) - 0.5f;
    const float hi = first_true(0.0f, far_hi, [&](float y) { return code_of(y, inv_so) == 127; }) + 0.5f;
    const float h = (hi - kLo) / (float)(t->nc - 1);
    // The cell boundaries are where fma(y, hinv, off) reaches an integer plus
    // 1/2 (the fma result is rounded to an integer next to kGeluBase), so
    // with an integer offset F, hinv = D / |y_min| for D an integer plus 1/2
    // puts a boundary at GELU's minimum y_min whatever F is. D is the
    // largest such value not above 1 / h: the cells widen by less than one
    // part in 2D, and still cover [kLo, hi]. When the minimum lies within
    // two cells of zero (large output scales, where every code near it is 0)
    // no boundary is placed there.
    double hinv = 1.0 / (double)h;
    const double D = floor(hinv * -kGeluMinY - 0.5) + 0.5;
    if (D >= 1.5) hinv = D / -kGeluMinY;
    t->hinv = (float)hinv;
    const float F = floorf(-kLo * t->hinv);
    t->off = kGeluBase + F;
    if (!(isfinite(t->hinv) && t->hinv > 0.0f && isfinite(t->off))) return;
    if (code_of(kLo, inv_so) != 0 || code_of(hi, inv_so) != 127) return;

    float start = -3.0e38f;
    for (int c = 0; c < t->nc; ++c) {
        // [start, end]: the fp32 values whose cell is c
        const float end = c + 1 < t->nc ? unord(ord(first_true(start, 3.0e38f, [&](float y) {
                                             return cell_of(*t, y) > c;
                                         })) - 1)
                                        : 3.0e38f;
        const float a = start < kLo ? kLo : start, b = end > hi ? hi : end;
        GeluCell &e = t->cell[c];
        if (a <= b && (double)b >= kGeluMinY - 0.5 * (double)h * 3 && (double)a <= kGeluMinY + 0.5 * (double)h * 3) {
            // the cells at the minimum: every fp32 value, unless the exact
            // values of the cell all round to one code with a margin far
            // above the fp32 expression's error
            if (!one_code_cell(a, b, inv_so, &e) && !exact_cell(a, b, inv_so, &e)) return;
        } else {
            const int q0 = code_of(a, inv_so), q1 = code_of(b, inv_so);
            e.q_lo = (int8_t)q0;
            e.q_hi = (int8_t)q1;
            e.pad = 0;
            if (q0 > q1 + 1 || q1 > q0 + 1) return;  // monotone: more than one change
            if (q0 == q1) {
                e.thr = INFINITY;
                // (monotone on this side of the minimum: no change inside;
                // a coarse scan guards the assumption)
                for (int sidx = 1; sidx < 32; ++sidx) {
                    const float y = a + (b - a) * ((float)sidx / 32.0f);
                    if (code_of(y, inv_so) != q0) return;
                }
            } else {
                const bool up = q1 > q0;
                const float thr = first_true(a, b, [&](float y) {
                    const int q = code_of(y, inv_so);
                    return up ? q >= q1 : q <= q1;
                });
                e.thr = thr;
                for (int sidx = 1; sidx < 32; ++sidx) {
                    const float y = a + (b - a) * ((float)sidx / 32.0f);
                    if (code_of(y, inv_so) != (y >= thr ? q1 : q0)) return;
                }
            }
        }
        start = unord(ord(end) + 1);
    }
    t->ok = true;
}

namespace {
// a fixed set of tables, one per recently used inverse output scale; a new
// scale takes the next slot round-robin
constexpr int kTableSlots = 32;
struct TableSlot {
    uint32_t key = 0;
    bool used = false;
    GeluTable t;
};
TableSlot g_slots[kTableSlots];
int g_next = 0;
std::mutex g_mu;
}  // namespace

bool gelu_table(float inv_so, GeluTable *out)
{
    uint32_t key;
    memcpy(&key, &inv_so, 4);
    std::lock_guard<std::mutex> lk(g_mu);
    for (TableSlot &sl : g_slots)
        if (sl.used && sl.key == key) {
            *out = sl.t;
            return out->ok;
        }
    TableSlot &sl = g_slots[g_next];
    g_next = (g_next + 1) % kTableSlots;
    sl.used = false;
    build(inv_so, &sl.t);
    sl.key = key;
    sl.used = true;
    *out = sl.t;
    return out->ok;
}

// The table's code for y, read exactly as the kernels read it: the cell from
// the clamped fma, then the threshold compare.
int gelu_table_code(const GeluTable &t, float y)
{
    const float cf = fmaxf(fminf(fmaf(y, t.hinv, t.off), kGeluBase + (float)(t.nc - 1)), kGeluBase);
    uint32_t bits;
    memcpy(&bits, &cf, 4);
    const GeluCell &e = t.cell[bits & 0xffffffu];
    return y >= e.thr ? e.q_hi : e.q_lo;
}

}  // namespace sl
