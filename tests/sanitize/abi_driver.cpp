// Test driver for the host side of the C ABI (include/buddy.h) under
// AddressSanitizer and UndefinedBehaviorSanitizer (test infrastructure
// only).  It is linked against the library's host code built with both
// sanitizers and calls only paths that never reach the device: argument
// validation of every entry point, the configuration checks of
// buddy_model_create (every rejected shape), the offline prior
// normalisation, the budget helper, and the launch-policy choice of a
// decode step.  Exit status 0 means every call returned the documented
// status and the sanitizers reported nothing.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "../../include/buddy.h"
#include "../../paper_2606_09514_amd/csrc/buddy_internal.h"

static int failures = 0;
#define EXPECT(cond, what)                                                   \
    do {                                                                     \
        if (!(cond)) { fprintf(stderr, "FAILED: %s (line %d)\n", what, __LINE__); ++failures; } \
    } while (0)

static buddy_config llama_like() {
    buddy_config c;
    memset(&c, 0, sizeof(c));
    c.n_layers = 32; c.d_model = 4096; c.n_heads = 32; c.n_kv_heads = 8; c.head_dim = 128;
    c.d_ffn = 14336; c.dm_hidden = 512; c.dm_act = BUDDY_ACT_SILU; c.dtype = BUDDY_BF16;
    c.max_batch = 4; c.max_ctx = 4096; c.rms_eps = 1e-5f; c.rope_theta = 5e5f;
    c.router_ctx = BUDDY_CTX_KV; c.start_layer = 1;
    return c;
}

int main() {
    // status strings and the budget helper
    for (int s = 0; s <= 7; ++s) EXPECT(buddy_status_string((buddy_status)s) != nullptr, "status");
    EXPECT(buddy_last_error(nullptr)[0] == '\0', "last_error(NULL)");
    EXPECT(buddy_budget_to_k(0.5f, 32) == 14, "budget 0.5");
    EXPECT(buddy_budget_to_k(1.0f, 32) == 30, "budget 1");
    EXPECT(buddy_budget_to_k(0.0f, 32) == -1 && buddy_budget_to_k(1.5f, 32) == -1, "budget range");
    EXPECT(buddy_budget_to_k(NAN, 32) == -1 && buddy_budget_to_k(0.5f, 1) == -1, "budget args");
    for (int L = 2; L < 300; L += 7)
        for (float b = 0.01f; b <= 1.0f; b += 0.01f) {
            const int k = buddy_budget_to_k(b, L);
            EXPECT(k >= 0 && k <= L - 2, "budget clamp");
        }

    // configuration checks: every rejection returns before any device call
    buddy_layer_weights lw[64];
    memset(lw, 0, sizeof(lw));
    int dummy = 0;
    for (int l = 0; l < 64; ++l)
        lw[l] = {&dummy, &dummy, &dummy, &dummy, &dummy, &dummy};
    buddy_dm_weights dm = {&dummy, &dummy, &dummy, &dummy, nullptr, 0.1f};
    buddy_model* m = (buddy_model*)&dummy;
    struct Case { void (*edit)(buddy_config&); buddy_status want; } cases[] = {
        {[](buddy_config& c) { c.n_layers = 1; }, BUDDY_ESHAPE},
        {[](buddy_config& c) { c.n_layers = 5000; }, BUDDY_ESHAPE},
        {[](buddy_config& c) { c.start_layer = 32; }, BUDDY_EINVAL},
        {[](buddy_config& c) { c.start_layer = -1; }, BUDDY_EINVAL},
        {[](buddy_config& c) { c.d_model = 4100; }, BUDDY_ESHAPE},
        {[](buddy_config& c) { c.n_heads = 30; }, BUDDY_ESHAPE},
        {[](buddy_config& c) { c.n_kv_heads = 2; }, BUDDY_ESHAPE},      // 16 heads per group
        {[](buddy_config& c) { c.n_kv_heads = 0; }, BUDDY_ESHAPE},
        {[](buddy_config& c) { c.head_dim = 96; }, BUDDY_ESHAPE},
        {[](buddy_config& c) { c.d_ffn = 0; }, BUDDY_ESHAPE},
        {[](buddy_config& c) { c.dm_hidden = 12; }, BUDDY_ESHAPE},
        {[](buddy_config& c) { c.dm_act = 7; }, BUDDY_EINVAL},
        {[](buddy_config& c) { c.dtype = 3; }, BUDDY_EINVAL},
        {[](buddy_config& c) { c.max_batch = 0; }, BUDDY_ECAPACITY},
        {[](buddy_config& c) { c.max_batch = 257; }, BUDDY_ECAPACITY},
        {[](buddy_config& c) { c.max_ctx = 0; }, BUDDY_EINVAL},
        {[](buddy_config& c) { c.max_ctx = (1 << 20) + 1; }, BUDDY_ECAPACITY},
        {[](buddy_config& c) { c.rope_theta = 0.f; }, BUDDY_EINVAL},
        {[](buddy_config& c) { c.rms_eps = NAN; }, BUDDY_EINVAL},
        {[](buddy_config& c) { c.router_ctx = 9; }, BUDDY_EINVAL},
        {[](buddy_config& c) { c.d_ffn = 40960; }, BUDDY_ESHAPE},       // activation row > LDS
        {[](buddy_config& c) { c.d_model = 8200; }, BUDDY_ESHAPE},
        {[](buddy_config& c) { c.dtype = BUDDY_F32; }, BUDDY_ESHAPE},   // fp32 rows too long
    };
    for (const Case& cs : cases) {
        buddy_config c = llama_like();
        cs.edit(c);
        m = (buddy_model*)&dummy;
        EXPECT(buddy_model_create(&c, lw, &dm, &m) == cs.want && m == nullptr, "config check");
    }
    {
        buddy_config c = llama_like();
        EXPECT(buddy_model_create(nullptr, lw, &dm, &m) == BUDDY_EINVAL, "null config");
        EXPECT(buddy_model_create(&c, nullptr, &dm, &m) == BUDDY_EINVAL, "null layers");
        EXPECT(buddy_model_create(&c, lw, nullptr, &m) == BUDDY_EINVAL, "null dm");
        EXPECT(buddy_model_create(&c, lw, &dm, nullptr) == BUDDY_EINVAL, "null out");
        lw[5].wdown = nullptr;
        EXPECT(buddy_model_create(&c, lw, &dm, &m) == BUDDY_EINVAL && !m, "null weight");
        lw[5].wdown = &dummy;
        buddy_dm_weights dm2 = dm;
        dm2.b2 = nullptr;
        EXPECT(buddy_model_create(&c, lw, &dm2, &m) == BUDDY_EINVAL && !m, "null dm weight");
    }

    // entry points without a handle, or with arguments rejected on the host
    buddy_kv kv;
    memset(&kv, 0, sizeof(kv));
    int32_t pos[2] = {0, 0}, ks[2] = {1, 1};
    float f = 0.f;
    uint8_t mk[4];
    EXPECT(buddy_decode_step(nullptr, &kv, &f, pos, ks, 1, 0, nullptr, nullptr, nullptr, nullptr) ==
               BUDDY_EINVAL, "decode without handle");
    EXPECT(buddy_pool_route(nullptr, &kv, pos, &f, 1, &f, nullptr) == BUDDY_EINVAL, "pool_route");
    EXPECT(buddy_predict_budget(nullptr, &kv, pos, &f, 1, pos, &f, nullptr) == BUDDY_EINVAL,
           "predict_budget");
    EXPECT(buddy_decode_step_auto(nullptr, &kv, &f, pos, 1, 0, pos, mk, &f, nullptr) ==
               BUDDY_EINVAL, "decode_auto");
    EXPECT(buddy_prefill(nullptr, &kv, &f, 1, pos, ks, 1, 0, nullptr, nullptr, nullptr, nullptr) ==
               BUDDY_EINVAL, "prefill");
    EXPECT(buddy_set_launch_policy(nullptr, 0) == BUDDY_EINVAL, "policy");
    EXPECT(buddy_set_gemm_tile(nullptr, 0) == BUDDY_EINVAL, "tile");
    EXPECT(buddy_set_budget_predictor(nullptr, nullptr) == BUDDY_EINVAL, "predictor");
    EXPECT(buddy_set_timing_events(nullptr, 0, 0, nullptr, nullptr, 0) == BUDDY_EINVAL, "timing");
    buddy_model_destroy(nullptr);
    EXPECT(buddy_select_topk(&f, ks, 0, 4, mk, nullptr) == BUDDY_OK, "topk B = 0");
    EXPECT(buddy_select_topk(nullptr, ks, 1, 4, mk, nullptr) == BUDDY_EINVAL, "topk scores");
    EXPECT(buddy_select_topk(&f, ks, 1, 0, mk, nullptr) == BUDDY_EINVAL, "topk n = 0");
    EXPECT(buddy_select_topk(&f, ks, 1, 256, mk, nullptr) == BUDDY_EINVAL, "topk n = 256");
    EXPECT(buddy_select_topk(&f, ks, 65536, 4, mk, nullptr) == BUDDY_EINVAL, "topk B");
    int32_t pi[4];
    EXPECT(buddy_group_by_route(mk, 0, 4, pi, pi, pi, nullptr) == BUDDY_OK, "group B = 0");
    EXPECT(buddy_group_by_route(nullptr, 1, 4, pi, pi, pi, nullptr) == BUDDY_EINVAL, "group mask");
    EXPECT(buddy_group_by_route(mk, 1, 0, pi, pi, pi, nullptr) == BUDDY_EINVAL, "group n = 0");
    EXPECT(buddy_group_by_route(mk, 1, 256, pi, pi, pi, nullptr) == BUDDY_EINVAL, "group n");
    EXPECT(buddy_group_by_route(mk, 1025, 4, pi, pi, pi, nullptr) == BUDDY_EINVAL, "group B");
    EXPECT(buddy_group_by_route(mk, 1, 4, nullptr, pi, pi, nullptr) == BUDDY_EINVAL, "group perm");
    int32_t kbad[1] = {5};
    EXPECT(buddy_select_topk(&f, kbad, 1, 4, mk, nullptr) == BUDDY_EINVAL, "topk k > n");

    // App. B prior normalisation (host code): every kind, winsorising, ties,
    // n = 1, and the documented rejections (nothing written on failure)
    const float raw[9] = {3.f, -1.f, 0.5f, 0.5f, 10.f, 0.f, 2.f, 0.5f, 1e-3f};
    float out[9];
    for (int kind = 0; kind < 3; ++kind)
        for (float w : {0.f, 1.5f}) {
            EXPECT(buddy_prior_normalize(raw, 9, kind, w, out) == BUDDY_OK, "prior");
            for (float v : out) EXPECT(isfinite(v), "prior finite");
            EXPECT(buddy_prior_normalize(raw, 1, kind, w, out) == BUDDY_OK, "prior n = 1");
        }
    for (float& v : out) v = 42.f;
    const float bad[2] = {1.f, NAN};
    EXPECT(buddy_prior_normalize(bad, 2, 0, 0.f, out) == BUDDY_EINVAL, "prior NaN");
    EXPECT(buddy_prior_normalize(raw, 0, 0, 0.f, out) == BUDDY_EINVAL, "prior n = 0");
    EXPECT(buddy_prior_normalize(raw, 9, 3, 0.f, out) == BUDDY_EINVAL, "prior kind");
    EXPECT(buddy_prior_normalize(raw, 9, 0, -1.f, out) == BUDDY_EINVAL, "prior winsor");
    EXPECT(buddy_prior_normalize(raw, 9, 0, INFINITY, out) == BUDDY_EINVAL, "prior winsor inf");
    EXPECT(buddy_prior_normalize(nullptr, 9, 0, 0.f, out) == BUDDY_EINVAL, "prior null");
    for (float v : out) EXPECT(v == 42.f, "nothing written on a rejection");

    // launch policy of a decode step's routable blocks (1 host-routed, 0
    // device-routed, -1 refused): under stream capture the automatic policy
    // never waits for the device and an explicit host-routed one is refused
    using buddy::choose_host_routed;
    using buddy::kHostRoutedMaxBatch;
    for (int cap = 0; cap < 2; ++cap)
        for (int all = 0; all < 2; ++all)
            for (int B : {1, kHostRoutedMaxBatch, kHostRoutedMaxBatch + 1, 256}) {
                const int a = choose_host_routed(BUDDY_LAUNCH_AUTO, all, B, 30, cap);
                EXPECT(a == (!cap && !all && B <= kHostRoutedMaxBatch ? 1 : 0), "auto policy");
                EXPECT(choose_host_routed(BUDDY_LAUNCH_DEVICE_ROUTED, all, B, 30, cap) == 0,
                       "device-routed policy");
                EXPECT(choose_host_routed(BUDDY_LAUNCH_HOST_ROUTED, all, B, 30, cap) ==
                           (cap ? -1 : 1), "host-routed policy");
                EXPECT(choose_host_routed(BUDDY_LAUNCH_HOST_ROUTED, all, B, 0, cap) == 0,
                       "no routable block");
            }

    if (failures) return 1;
    printf("abi driver ok\n");
    return 0;
}
