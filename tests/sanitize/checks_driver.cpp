// checks_driver.cpp -- exercises the C ABI's host-side argument checks
// (paper_2608_23048_amd/csrc/checks.cpp) under the host compiler's address and
// undefined-behaviour sanitizers: every case states the status it expects.
// Pointers are fake addresses that are never dereferenced.
#include "checks.hpp"

#include <cstdio>
#include <cstdlib>
#include <vector>

using namespace roi;

static int failures = 0;

static void expect(const char* what, int got, int want)
{
    if (got != want) {
        std::printf("FAIL %s: status %d, expected %d (%s)\n", what, got, want,
                    g_last_error.c_str());
        ++failures;
    }
}

template <typename T>
static T* fake(uintptr_t a) { return reinterpret_cast<T*>(a); }

static roi_fwd_tensor fwd_tensor(uintptr_t base, int64_t rows, int64_t cols, uint64_t off,
                                 bool s, bool idx)
{
    roi_fwd_tensor t{};
    t.W = fake<const uint16_t>(base);
    t.logits = fake<const float>(base + (1ull << 32));
    t.rows = rows;
    t.cols = cols;
    t.elem_offset = off;
    t.W_masked = fake<uint16_t>(base + (2ull << 32));
    t.soft_mask = s ? fake<float>(base + (3ull << 32)) : nullptr;
    t.sel_idx = idx ? fake<uint8_t>(base + (4ull << 32)) : nullptr;
    return t;
}

int main()
{
    const uintptr_t B = 0x100000000000ull;
    int ws, wi;
    // patterns, sizes, temperatures
    expect("4:4", check_common(4, 4, 1.0f, 1.0f), ROI_OK);
    expect("32:32", check_common(32, 32, 1.0f, 1.0f), ROI_OK);
    expect("0:4", check_common(0, 4, 1.0f, 1.0f), ROI_E_INVAL);
    expect("5:4", check_common(5, 4, 1.0f, 1.0f), ROI_E_INVAL);
    expect("2:6", check_common(2, 6, 1.0f, 1.0f), ROI_E_UNSUPPORTED);
    expect("2:64", check_common(2, 64, 1.0f, 1.0f), ROI_E_UNSUPPORTED);
    expect("tau 0", check_common(2, 4, 0.0f, 1.0f), ROI_E_INVAL);
    expect("tau nan", check_common(2, 4, __builtin_nanf(""), 1.0f), ROI_E_INVAL);
    expect("lambda inf", check_common(2, 4, 1.0f, __builtin_inff()), ROI_E_INVAL);
    Shape sh;
    expect("empty", check_shape(0, 0, 2, 4, 1.0f, 1.0f, 0, &sh), ROI_OK);
    expect("one group", check_shape(1, 4, 2, 4, 1.0f, 1.0f, 0, &sh), ROI_OK);
    expect("rows < 0", check_shape(-1, 4, 2, 4, 1.0f, 1.0f, 0, &sh), ROI_E_INVAL);
    expect("cols % m", check_shape(2, 6, 2, 4, 1.0f, 1.0f, 0, &sh), ROI_E_INVAL);
    expect("2^62", check_shape((int64_t)1 << 31, (int64_t)1 << 31, 2, 4, 1.0f, 1.0f, 0, &sh),
           ROI_E_INVAL);
    expect("below 2^62", check_shape((int64_t)1 << 30, (int64_t)1 << 31, 2, 4, 1.0f, 1.0f, 0, &sh),
           ROI_OK);
    expect("offset % m", check_shape(1, 32, 2, 32, 1.0f, 1.0f, 16, &sh), ROI_E_INVAL);
    expect("offset overflow", check_shape(1, 8, 2, 4, 1.0f, 1.0f, UINT64_MAX - 3, &sh),
           ROI_E_INVAL);
    expect("offset at the top", check_shape(1, 4, 2, 4, 1.0f, 1.0f, UINT64_MAX - 3 - 4, &sh),
           ROI_OK);
    expect("count < 0", check_count(nullptr, -1), ROI_E_INVAL);
    expect("count 0, NULL", check_count(nullptr, 0), ROI_OK);
    expect("count 1, NULL", check_count(nullptr, 1), ROI_E_INVAL);

    // overlaps: inputs may overlap inputs; an output overlaps nothing
    {
        std::vector<Range> r;
        add_range(r, fake<void>(B), 64, false);
        add_range(r, fake<void>(B + 32), 64, false);
        add_range(r, fake<void>(B + 96), 16, true); // adjacent, not overlapping
        expect("inputs overlap inputs", check_overlaps(r), ROI_OK);
        add_range(r, fake<void>(B + 100), 4, true);
        expect("outputs overlap", check_overlaps(r), ROI_E_INVAL);
        std::vector<Range> q;
        add_range(q, fake<void>(B + 8), 8, false);
        add_range(q, fake<void>(B), 64, true);
        expect("input inside an output", check_overlaps(q), ROI_E_INVAL);
        std::vector<Range> z;
        add_range(z, nullptr, 64, true);
        add_range(z, fake<void>(B), 0, true);
        expect("empty ranges are skipped", check_overlaps(z), ROI_OK);
        expect("overlap()", overlap(fake<void>(B), 16, fake<void>(B + 15), 1), true);
        expect("no overlap()", overlap(fake<void>(B), 16, fake<void>(B + 16), 1), false);
    }

    // forward descriptors
    {
        roi_fwd_tensor t[3] = {fwd_tensor(B, 4, 8, 0, true, true),
                               fwd_tensor(B + (8ull << 32), 0, 8, 32, false, false),
                               fwd_tensor(B + (16ull << 32), 2, 32, 32, true, true)};
        expect("fwd ok", validate_fwd(t, 3, 2, 4, 1.0f, 1.0f, &ws, &wi), ROI_OK);
        expect("fwd flags", ws == 1 && wi == 1, true);
        expect("fwd count 0", validate_fwd(nullptr, 0, 2, 4, 1.0f, 1.0f, &ws, &wi), ROI_OK);
        expect("fwd nothing to do", ws, -1);
        roi_fwd_tensor e = fwd_tensor(0, 0, 4, 0, false, false);
        e.W = nullptr;
        e.logits = nullptr;
        e.W_masked = nullptr;
        expect("fwd empty NULL tensor", validate_fwd(&e, 1, 2, 4, 1.0f, 1.0f, &ws, &wi), ROI_OK);
        roi_fwd_tensor u = t[0];
        u.logits = fake<const float>(B + 4);
        expect("fwd misaligned", validate_fwd(&u, 1, 2, 4, 1.0f, 1.0f, &ws, &wi), ROI_E_INVAL);
        u = t[0];
        u.W_masked = nullptr;
        expect("fwd NULL output", validate_fwd(&u, 1, 2, 4, 1.0f, 1.0f, &ws, &wi), ROI_E_INVAL);
        u = t[0];
        u.soft_mask = fake<float>(B + (1ull << 32) + 16); // inside the logits
        expect("fwd S over logits", validate_fwd(&u, 1, 2, 4, 1.0f, 1.0f, &ws, &wi), ROI_E_INVAL);
        roi_fwd_tensor mix[2] = {t[0], fwd_tensor(B + (8ull << 32), 2, 8, 64, false, true)};
        expect("fwd mixed S", validate_fwd(mix, 2, 2, 4, 1.0f, 1.0f, &ws, &wi), ROI_E_INVAL);
        roi_fwd_tensor two[2] = {t[0], t[0]};
        expect("fwd two calls' outputs overlap", validate_fwd(two, 2, 2, 4, 1.0f, 1.0f, &ws, &wi),
               ROI_E_INVAL);
        roi_fwd_tensor bad = fwd_tensor(B, 3, 30, 0, false, false);
        expect("fwd tensor shape", validate_fwd(&bad, 1, 2, 4, 1.0f, 1.0f, &ws, &wi), ROI_E_INVAL);
    }

    // backward descriptors, with and without the AdamW step
    {
        BwdDesc d{fake<const uint16_t>(B), fake<const uint16_t>(B + (1ull << 32)),
                  fake<const float>(B + (2ull << 32)), fake<float>(B + (3ull << 32)),
                  nullptr, nullptr, 64, 32, 0};
        AdamStep st{};
        bool any;
        expect("bwd ok", validate_bwd(&d, 1, 16, 32, 1.0f, 1.0f, nullptr, &st, &any), ROI_OK);
        expect("bwd any", any, true);
        BwdDesc e = d;
        e.dphi = fake<float>(B + 16); // inside grad_W_masked
        expect("bwd output over input", validate_bwd(&e, 1, 2, 4, 1.0f, 1.0f, nullptr, &st, &any),
               ROI_E_INVAL);
        roi_adamw_params o{1e-3f, 0.9f, 0.95f, 1e-8f, 0.05f, 4};
        BwdDesc a = d;
        a.dphi = nullptr;
        a.m = fake<float>(B + (4ull << 32));
        a.v = fake<float>(B + (5ull << 32));
        expect("adamw ok", validate_bwd(&a, 1, 2, 4, 1.0f, 1.0f, &o, &st, &any), ROI_OK);
        expect("adamw step size", st.step_size > 0.0f && st.inv_sqrt_bc2 > 1.0f, true);
        a.v = nullptr;
        expect("adamw NULL moment", validate_bwd(&a, 1, 2, 4, 1.0f, 1.0f, &o, &st, &any),
               ROI_E_INVAL);
        roi_adamw_params b = o;
        b.beta2 = 1.0f;
        expect("adamw beta2 = 1", check_adamw(&b, &st), ROI_E_INVAL);
        b = o;
        b.t = 0;
        expect("adamw t = 0", check_adamw(&b, &st), ROI_E_INVAL);
        expect("adamw NULL", check_adamw(nullptr, &st), ROI_E_INVAL);
        expect("bwd count < 0", validate_bwd(&d, -1, 2, 4, 1.0f, 1.0f, nullptr, &st, &any),
               ROI_E_INVAL);
    }

    // the categorical sampler: C = binom(m, n) logits per group
    {
        int64_t ng;
        int C;
        const uint16_t* W = fake<const uint16_t>(B);
        const float* A = fake<const float>(B + (1ull << 32));
        uint16_t* Wm = fake<uint16_t>(B + (8ull << 32));
        float* dA = fake<float>(B + (9ull << 32));
        const uint16_t* G = fake<const uint16_t>(B + (10ull << 32));
        expect("cat 4:8", validate_cat(true, W, A, nullptr, 3, 8, 4, 8, 1.0f, 1.0f, 0, Wm, nullptr,
                                       nullptr, nullptr, &ng, &C), ROI_OK);
        expect("cat 4:8 sizes", ng == 3 && C == 70, true);
        expect("cat 8:8", validate_cat(false, W, A, G, 1, 8, 8, 8, 1.0f, 1.0f, 0, nullptr, nullptr,
                                       nullptr, dA, &ng, &C), ROI_OK);
        expect("cat 8:8 one candidate", C, 1);
        expect("cat m = 16", validate_cat(true, W, A, nullptr, 1, 16, 2, 16, 1.0f, 1.0f, 0, Wm,
                                          nullptr, nullptr, nullptr, &ng, &C), ROI_E_UNSUPPORTED);
        // 2^57 groups of 70 logits: 4 * 70 * 2^57 bytes do not fit in 2^62
        expect("cat logits bytes", validate_cat(true, W, A, nullptr, (int64_t)1 << 30,
                                                (int64_t)1 << 30, 4, 8, 1.0f, 1.0f, 0, Wm,
                                                nullptr, nullptr, nullptr, &ng, &C), ROI_E_INVAL);
        expect("cat noise index overflow",
               validate_cat(true, W, A, nullptr, 1, 8, 4, 8, 1.0f, 1.0f, UINT64_MAX / 8, Wm,
                            nullptr, nullptr, nullptr, &ng, &C), ROI_E_INVAL);
        expect("cat dalpha over alpha",
               validate_cat(false, W, A, G, 2, 8, 2, 4, 1.0f, 1.0f, 0, nullptr, nullptr, nullptr,
                            const_cast<float*>(A) + 4, &ng, &C), ROI_E_INVAL);
        expect("cat empty", validate_cat(false, nullptr, nullptr, nullptr, 0, 8, 2, 4, 1.0f, 1.0f,
                                         0, nullptr, nullptr, nullptr, nullptr, &ng, &C), ROI_OK);
    }

    // pieces: the high 32 bits of every Philox block index are the same
    // within a piece, and the pieces tile the range exactly
    for (int64_t per : {4, 8, 16, 32}) {
        const uint64_t starts[] = {0, ((uint64_t)1 << 34) - (uint64_t)per * 3,
                                   ((uint64_t)5 << 34) - (uint64_t)per, UINT64_MAX / 2 + 1};
        for (uint64_t off : starts) {
            const int64_t items = ((int64_t)1 << 32) + 7;
            int64_t next = 0;
            const int st = for_each_piece(off, items, per, [&](int64_t g0, int64_t n, uint64_t e0) {
                if (g0 != next || n < 1 || e0 != off + (uint64_t)g0 * (uint64_t)per) return 1;
                const uint64_t first = e0 / 4, last = (e0 + (uint64_t)(n * per) - 1) / 4;
                if ((first >> 32) != (last >> 32)) return 2;
                next = g0 + n;
                return 0;
            });
            expect("pieces", st, 0);
            expect("pieces cover the range", next == items, true);
        }
    }
    expect("error text set by a failure", check_common(0, 4, 1.0f, 1.0f) != ROI_OK &&
                                              !g_last_error.empty(), true);
    expect("ok() clears it", ok() == ROI_OK && g_last_error.empty(), true);
    if (failures) return 1;
    std::printf("checks ok\n");
    return 0;
}
