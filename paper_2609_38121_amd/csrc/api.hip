// Host-side pieces of the WUSH-KV C ABI shared by every entry point:
// descriptor validation, status strings, sizes, and the opt-in kernel timer.
#include <cmath>
#include <cstring>
#include <vector>

#include "common.h"

namespace wushkv {

namespace {

struct Timing {
    std::vector<hipEvent_t> ev;        // 2 per slot: start, stop
    std::vector<const char *> names;   // per slot
    int slots = 0;
    int used = 0;
};
Timing g_timing;

}  // namespace

TimedLaunch timing_slot(const char *name)
{
    Timing &t = g_timing;
    if (t.slots == 0 || t.used >= t.slots) return TimedLaunch{};
    t.names[t.used] = name;
    const TimedLaunch r{t.ev[2 * t.used], t.ev[2 * t.used + 1]};
    t.used += 1;
    return r;
}

}  // namespace wushkv

using namespace wushkv;

static bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int wushkv_validate_cache(const wushkv_cache *c)
{
    if (c == nullptr) return WUSHKV_EINVAL;
    if (c->batch < 1 || c->n_kv_heads < 1) return WUSHKV_EINVAL;
    if (c->head_dim != 64 && c->head_dim != 128) return WUSHKV_EUNSUPPORTED;
    if (c->bits < 2 || c->bits > 4) return WUSHKV_EUNSUPPORTED;
    if (c->s_sink < 0 || c->s_keep < 0 || c->s_flush < 1) return WUSHKV_EINVAL;
    if (c->win_slots < kPage || c->win_slots % kPage != 0) return WUSHKV_EINVAL;
    const int64_t need = (int64_t)c->s_keep + c->s_flush - 1;
    const int64_t ring = (int64_t)c->win_slots - c->s_sink;
    if (ring < 1 || ring < need) return WUSHKV_EINVAL;
    if (c->max_pages_per_seq < 0 || c->n_pages < 0) return WUSHKV_EINVAL;
    if (c->codec == WUSHKV_CODEC_PCLIP) {
        if (!(c->kappa_k > 0.0f && c->kappa_k <= 1.0f)) return WUSHKV_EINVAL;
        if (!(c->kappa_v > 0.0f && c->kappa_v <= 1.0f)) return WUSHKV_EINVAL;
    } else if (c->codec == WUSHKV_CODEC_QUEST) {
        if (!(c->quest_alpha > 0.0f && c->quest_alpha < INFINITY)) return WUSHKV_EINVAL;
    } else {
        return WUSHKV_EINVAL;
    }
    if (!c->win_k || !c->win_v || !c->seq_len || !c->quant_end || !c->commit) return WUSHKV_EINVAL;
    const bool paged = c->n_pages > 0 && c->max_pages_per_seq > 0;
    if (paged && (!c->pages || !c->page_table)) return WUSHKV_EINVAL;
    if (!aligned16(c->win_k) || !aligned16(c->win_v) || !aligned16(c->pages) ||
        !aligned16(c->page_table) || !aligned16(c->seq_len) || !aligned16(c->quant_end) ||
        !aligned16(c->commit))
        return WUSHKV_EINVAL;
    // every element offset the kernels form must fit in int64 with margin
    const double win = (double)c->batch * c->n_kv_heads * c->win_slots * c->head_dim;
    const double pool = (double)c->n_pages * c->n_kv_heads *
                        (double)wushkv_page_bytes(c->head_dim, c->bits);
    if (win > 9.0e15 || pool > 9.0e15) return WUSHKV_EINVAL;
    return WUSHKV_OK;
}

extern "C" size_t wushkv_page_bytes(int32_t head_dim, int32_t bits)
{
    if ((head_dim != 64 && head_dim != 128) || bits < 2 || bits > 4) return 0;
    return (size_t)kPage * (2 * head_dim * storage_bits(bits) / 8 + 8);
}

extern "C" const char *wushkv_status_string(int status)
{
    switch (status) {
        case WUSHKV_OK: return "ok";
        case WUSHKV_EINVAL: return "invalid argument";
        case WUSHKV_EUNSUPPORTED: return "unsupported configuration";
        case WUSHKV_EWORKSPACE: return "workspace too small";
        case WUSHKV_ELAUNCH: return "kernel launch failed";
        case WUSHKV_ENODEVICE: return "no usable device";
    }
    return "unknown status";
}

extern "C" int wushkv_abi_version(void) { return WUSHKV_ABI_VERSION; }

namespace {

// Standard normal density and the probability of [a, b), 0 <= a <= b <= inf.
double npdf(double x) { return std::isinf(x) ? 0.0 : 0.3989422804014327 * std::exp(-0.5 * x * x); }
double nprob(double a, double b) { return 0.5 * (std::erfc(a * M_SQRT1_2) - std::erfc(b * M_SQRT1_2)); }

// E[zh^2] - E[z zh] for zh the level nearest to a standard Gaussian z on the
// grid of n = 2^bits levels from -alpha to alpha (levels (k + 1/2) step, step
// 2 alpha / (n - 1), bin [k step, (k + 1) step), outer bins unbounded).
// Every level scales with alpha and the bins are the nearest-level cells, so
// the derivative of the mean squared error in alpha is 2 / alpha times this
// value: the optimum is its root.  By symmetry only the bins above zero are
// summed (and doubled).
double quest_gradient(int bits, double alpha)
{
    const int half = 1 << (bits - 1);
    const double step = 2.0 * alpha / (2.0 * half - 1.0);
    double g = 0.0;
    for (int k = 0; k < half; ++k) {
        const double a = k * step;
        const double b = (k == half - 1) ? INFINITY : (k + 1) * step;
        const double lvl = (k + 0.5) * step;
        g += lvl * lvl * nprob(a, b) - lvl * (npdf(a) - npdf(b));
    }
    return 2.0 * g;
}

}  // namespace

extern "C" double wushkv_quest_alpha(int32_t bits)
{
    if (bits < 1 || bits > 8) return NAN;
    // the gradient is negative below the optimum and positive above it
    double lo = 1e-3, hi = 16.0;
    for (int it = 0; it < 200 && hi - lo > 1e-15 * hi; ++it) {
        const double mid = 0.5 * (lo + hi);
        if (quest_gradient(bits, mid) < 0.0) lo = mid;
        else hi = mid;
    }
    return 0.5 * (lo + hi);
}

extern "C" int wushkv_timing_enable(int32_t slots)
{
    Timing &t = g_timing;
    for (hipEvent_t e : t.ev) (void)hipEventDestroy(e);
    t.ev.clear();
    t.names.clear();
    t.slots = 0;
    t.used = 0;
    if (slots <= 0) return WUSHKV_OK;
    if (slots > (1 << 20)) return WUSHKV_EINVAL;
    t.ev.resize(2 * (size_t)slots);
    t.names.resize(slots, nullptr);
    for (size_t i = 0; i < t.ev.size(); ++i) {
        if (hipEventCreate(&t.ev[i]) != hipSuccess) {
            t.ev.resize(i);
            wushkv_timing_enable(0);
            return WUSHKV_ENODEVICE;
        }
    }
    t.slots = slots;
    return WUSHKV_OK;
}

extern "C" int wushkv_timing_read(const char *name_substr, int32_t *count, double *total_ms)
{
    Timing &t = g_timing;
    if (!count || !total_ms) return WUSHKV_EINVAL;
    *count = 0;
    *total_ms = 0.0;
    for (int i = 0; i < t.used; ++i) {
        if (name_substr && !std::strstr(t.names[i], name_substr)) continue;
        if (hipEventSynchronize(t.ev[2 * i + 1]) != hipSuccess) return WUSHKV_ELAUNCH;
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, t.ev[2 * i], t.ev[2 * i + 1]) != hipSuccess)
            return WUSHKV_ELAUNCH;
        *count += 1;
        *total_ms += ms;
    }
    return WUSHKV_OK;
}

extern "C" int wushkv_timing_launch(int32_t index, const char **name, double *ms)
{
    Timing &t = g_timing;
    if (!name || !ms || index < 0 || index >= t.used) return WUSHKV_EINVAL;
    if (hipEventSynchronize(t.ev[2 * index + 1]) != hipSuccess) return WUSHKV_ELAUNCH;
    float f = 0.0f;
    if (hipEventElapsedTime(&f, t.ev[2 * index], t.ev[2 * index + 1]) != hipSuccess) return WUSHKV_ELAUNCH;
    *name = t.names[index];
    *ms = f;
    return WUSHKV_OK;
}

extern "C" int wushkv_timing_count(void) { return g_timing.used; }
