// checks.cpp -- the host-side argument checks of the C ABI (checks.hpp).
#include "checks.hpp"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>

namespace roi {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return status;
}

int ok()
{
    g_last_error.clear();
    return ROI_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool overlap(const void* a, size_t na, const void* b, size_t nb)
{
    if (!a || !b || na == 0 || nb == 0) return false;
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + nb && b0 < a0 + na;
}

// Sorted by start, a range overlaps an earlier one exactly when it starts
// before the largest end seen so far (of any range, for an output; of the
// outputs, for an input).
int check_overlaps(std::vector<Range>& r)
{
    std::sort(r.begin(), r.end(), [](const Range& a, const Range& b) { return a.p < b.p; });
    uintptr_t end_any = 0, end_out = 0;
    for (const Range& x : r) {
        if (x.out ? x.p < end_any : x.p < end_out)
            return fail(ROI_E_INVAL, "an output overlaps another input or output");
        end_any = std::max(end_any, x.p + x.n);
        if (x.out) end_out = std::max(end_out, x.p + x.n);
    }
    return ROI_OK;
}

void add_range(std::vector<Range>& r, const void* p, size_t n, bool out)
{
    if (p && n) r.push_back({(uintptr_t)p, n, out});
}

int check_common(int n, int m, float tau, float lambda)
{
    if (m < 1 || n < 1 || n > m)
        return fail(ROI_E_INVAL, "pattern n:m = %d:%d needs 1 <= n <= m", n, m);
    if (m != 4 && m != 8 && m != 16 && m != 32)
        return fail(ROI_E_UNSUPPORTED, "m = %d is not built (supported: 4, 8, 16, 32)", m);
    if (!(tau > 0.0f) || !std::isfinite(tau))
        return fail(ROI_E_INVAL, "tau must be finite and > 0");
    if (!(lambda > 0.0f) || !std::isfinite(lambda))
        return fail(ROI_E_INVAL, "lambda must be finite and > 0");
    return ROI_OK;
}

int check_shape(int64_t rows, int64_t cols, int n, int m, float tau, float lambda,
                uint64_t elem_offset, Shape* sh)
{
    if (rows < 0 || cols < 0) return fail(ROI_E_INVAL, "rows (%lld) and cols (%lld) must be >= 0",
                                          (long long)rows, (long long)cols);
    if (int st = check_common(n, m, tau, lambda)) return st;
    if (cols % m != 0) return fail(ROI_E_INVAL, "cols (%lld) must be a multiple of m (%d)",
                                   (long long)cols, m);
    // rows * cols >= 2^62 exactly when cols > (2^62 - 1) / rows (integer division);
    // below it, the byte sizes of fp32 arrays (4 rows cols) fit in 64 bits
    if (rows > 0 && cols > (((int64_t)1 << 62) - 1) / rows)
        return fail(ROI_E_INVAL, "rows * cols must be below 2^62");
    if (elem_offset % (uint64_t)m != 0)
        return fail(ROI_E_INVAL, "elem_offset (%llu) must be a multiple of m (%d)",
                    (unsigned long long)elem_offset, m);
    const int64_t numel = rows * cols;
    if (elem_offset > UINT64_MAX - (uint64_t)numel)
        return fail(ROI_E_INVAL, "elem_offset + rows * cols overflows 64 bits");
    sh->numel = numel;
    sh->ngroups = numel / m;
    return ROI_OK;
}

int check_count(const void* t, int count)
{
    if (count < 0) return fail(ROI_E_INVAL, "count must be >= 0");
    if (count > 0 && !t) return fail(ROI_E_INVAL, "tensors must not be NULL");
    return ROI_OK;
}

int check_adamw(const roi_adamw_params* o, AdamStep* st)
{
    if (!o) return fail(ROI_E_INVAL, "the AdamW parameters must not be NULL");
    if (!(o->lr >= 0.0f) || !std::isfinite(o->lr))
        return fail(ROI_E_INVAL, "AdamW lr must be finite and >= 0");
    if (!(o->beta1 >= 0.0f && o->beta1 < 1.0f) || !(o->beta2 >= 0.0f && o->beta2 < 1.0f))
        return fail(ROI_E_INVAL, "AdamW betas must lie in [0, 1)");
    if (!(o->eps > 0.0f) || !std::isfinite(o->eps))
        return fail(ROI_E_INVAL, "AdamW eps must be finite and > 0");
    if (!(o->weight_decay >= 0.0f) || !std::isfinite(o->weight_decay))
        return fail(ROI_E_INVAL, "AdamW weight_decay must be finite and >= 0");
    if (o->t < 1) return fail(ROI_E_INVAL, "AdamW step count t must be >= 1");
    const double lr = o->lr, b1 = o->beta1, b2 = o->beta2;
    const double bc1 = 1.0 - std::pow(b1, (double)o->t);
    const double bc2 = 1.0 - std::pow(b2, (double)o->t);
    st->decay = (float)(1.0 - lr * (double)o->weight_decay);
    st->beta1 = o->beta1;
    st->beta2 = o->beta2;
    st->one_m_beta1 = (float)(1.0 - b1);
    st->one_m_beta2 = (float)(1.0 - b2);
    st->step_size = (float)(lr / bc1);
    st->inv_sqrt_bc2 = (float)(1.0 / std::sqrt(bc2));
    st->eps = o->eps;
    return ROI_OK;
}

int validate_fwd(const roi_fwd_tensor* t, int count, int n, int m, float tau, float lambda,
                 int* with_s, int* with_idx)
{
    *with_s = *with_idx = -1; // -1: no nonempty tensor seen yet
    if (int st = check_common(n, m, tau, lambda)) return st;
    if (int st = check_count(t, count)) return st;
    std::vector<Range> ranges;
    for (int i = 0; i < count; ++i) {
        Shape sh;
        if (int st = check_shape(t[i].rows, t[i].cols, n, m, tau, lambda, t[i].elem_offset, &sh))
            return count > 1 ? fail(st, "tensor %d: %s", i, g_last_error.c_str()) : st;
        if (sh.numel == 0) continue;
        if (!t[i].W || !t[i].logits || !t[i].W_masked)
            return fail(ROI_E_INVAL, "tensor %d: W, logits and W_masked must not be NULL", i);
        if (!aligned16(t[i].W) || !aligned16(t[i].logits) || !aligned16(t[i].W_masked) ||
            (t[i].soft_mask && !aligned16(t[i].soft_mask)) ||
            (t[i].sel_idx && !aligned16(t[i].sel_idx)))
            return fail(ROI_E_INVAL, "tensor %d: device pointers must be 16-byte aligned", i);
        const int s_i = t[i].soft_mask != nullptr, x_i = t[i].sel_idx != nullptr;
        if ((*with_s >= 0 && s_i != *with_s) || (*with_idx >= 0 && x_i != *with_idx))
            return fail(ROI_E_INVAL,
                        "soft_mask and sel_idx must each be given for every tensor or for none");
        *with_s = s_i;
        *with_idx = x_i;
        const size_t nb2 = (size_t)sh.numel * 2, nb4 = (size_t)sh.numel * 4;
        add_range(ranges, t[i].W, nb2, false);
        add_range(ranges, t[i].logits, nb4, false);
        add_range(ranges, t[i].W_masked, nb2, true);
        add_range(ranges, t[i].soft_mask, nb4, true);
        add_range(ranges, t[i].sel_idx, (size_t)sh.ngroups * (size_t)n, true);
    }
    if (*with_s < 0) return ok(); // nothing to do
    if (int st = check_overlaps(ranges)) return st;
    return ok();
}

int validate_bwd(const BwdDesc* t, int count, int n, int m, float tau, float lambda,
                 const roi_adamw_params* opt, AdamStep* astep, bool* any)
{
    *any = false;
    if (int st = check_common(n, m, tau, lambda)) return st;
    const bool adam = opt != nullptr;
    if (adam)
        if (int st = check_adamw(opt, astep)) return st;
    if (int st = check_count(t, count)) return st;
    std::vector<Range> ranges;
    for (int i = 0; i < count; ++i) {
        Shape sh;
        if (int st = check_shape(t[i].rows, t[i].cols, n, m, tau, lambda, t[i].off, &sh))
            return count > 1 ? fail(st, "tensor %d: %s", i, g_last_error.c_str()) : st;
        if (sh.numel == 0) continue;
        if (!t[i].G || !t[i].W || !t[i].phi || (!adam && !t[i].dphi) ||
            (adam && (!t[i].m || !t[i].v)))
            return fail(ROI_E_INVAL, adam ? "tensor %d: grad_W_masked, W, logits, exp_avg and "
                                            "exp_avg_sq must not be NULL"
                                          : "tensor %d: grad_W_masked, W, logits and grad_logits "
                                            "must not be NULL", i);
        if (!aligned16(t[i].G) || !aligned16(t[i].W) || !aligned16(t[i].phi) ||
            (t[i].dphi && !aligned16(t[i].dphi)) || (t[i].m && !aligned16(t[i].m)) ||
            (t[i].v && !aligned16(t[i].v)))
            return fail(ROI_E_INVAL, "tensor %d: device pointers must be 16-byte aligned", i);
        const size_t nb2 = (size_t)sh.numel * 2, nb4 = (size_t)sh.numel * 4;
        add_range(ranges, t[i].G, nb2, false);
        add_range(ranges, t[i].W, nb2, false);
        add_range(ranges, t[i].phi, nb4, adam); // updated in place by the AdamW step
        add_range(ranges, t[i].dphi, nb4, true);
        if (adam) {
            add_range(ranges, t[i].m, nb4, true);
            add_range(ranges, t[i].v, nb4, true);
        }
        *any = true;
    }
    if (!*any) return ok();
    if (int st = check_overlaps(ranges)) return st;
    return ok();
}

int validate_cat(bool fwd, const uint16_t* W, const float* alpha, const uint16_t* G, int64_t rows,
                 int64_t cols, int n, int m, float tau, float lambda, uint64_t group_offset,
                 const uint16_t* W_masked, const float* S, const uint8_t* choice,
                 const float* dalpha, int64_t* ngroups_out, int* C_out)
{
    *ngroups_out = 0;
    *C_out = 0;
    if (rows < 0 || cols < 0) return fail(ROI_E_INVAL, "rows and cols must be >= 0");
    if (m < 1 || n < 1 || n > m)
        return fail(ROI_E_INVAL, "pattern n:m = %d:%d needs 1 <= n <= m", n, m);
    if (m != 4 && m != 8)
        return fail(ROI_E_UNSUPPORTED, "the categorical sampler is built for m = 4 and 8");
    if (cols % m != 0) return fail(ROI_E_INVAL, "cols must be a multiple of m");
    if (rows > 0 && cols > (((int64_t)1 << 62) - 1) / rows)
        return fail(ROI_E_INVAL, "rows * cols must be below 2^62");
    if (!(tau > 0.0f) || !std::isfinite(tau)) return fail(ROI_E_INVAL, "tau must be finite, > 0");
    if (!(lambda > 0.0f) || !std::isfinite(lambda))
        return fail(ROI_E_INVAL, "lambda must be finite and > 0");
    int C = 1; // binom(m, n)
    for (int k = 1; k <= n; ++k) C = C * (m - n + k) / k;
    const int64_t ngroups = rows * cols / m;
    // the logits and their gradient hold 4 C bytes per group
    if (ngroups > ((int64_t)1 << 62) / (4 * (int64_t)C))
        return fail(ROI_E_INVAL, "the %d logits per group of %lld groups exceed 2^62 bytes", C,
                    (long long)ngroups);
    const uint64_t B = (uint64_t)(C + 3) / 4;
    if (ngroups > 0 && group_offset > (UINT64_MAX / (4 * B)) - (uint64_t)ngroups)
        return fail(ROI_E_INVAL, "group_offset + groups overflows the noise index space");
    *ngroups_out = ngroups;
    *C_out = C;
    if (ngroups == 0) return ok();
    if (!W || !alpha || (fwd ? !W_masked : (!G || !dalpha)))
        return fail(ROI_E_INVAL, "a required pointer is NULL");
    const void* ptrs[] = {W, alpha, G, W_masked, S, choice, dalpha};
    for (const void* p : ptrs)
        if (p && !aligned16(p)) return fail(ROI_E_INVAL, "device pointers must be 16-byte aligned");
    const size_t numel = (size_t)ngroups * (size_t)m, nc = (size_t)ngroups * (size_t)C;
    std::vector<Range> r;
    add_range(r, W, numel * 2, false);
    add_range(r, alpha, nc * 4, false);
    add_range(r, G, numel * 2, false);
    add_range(r, W_masked, numel * 2, true);
    add_range(r, S, numel * 4, true);
    add_range(r, choice, (size_t)ngroups, true);
    add_range(r, dalpha, nc * 4, true);
    if (int st = check_overlaps(r)) return st;
    return ok();
}

} // namespace roi
