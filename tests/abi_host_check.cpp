// Host-side driver of the C ABI for the sanitizer build (AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code of the library): every entry
// point that does not need a GPU, with valid arguments, the documented error
// cases and boundary values.  Prints one line per failed expectation and
// exits with the number of failures (0 = all as documented).
#include "../include/normpre.h"

#include <cmath>
#include <cstdio>
#include <cstring>
#include <vector>

static int failures = 0;

#define EXPECT(cond)                                                         \
    do {                                                                     \
        if (!(cond)) {                                                       \
            std::printf("FAILED line %d: %s\n", __LINE__, #cond);            \
            ++failures;                                                      \
        }                                                                    \
    } while (0)

int main() {
    normpre_hparams hp;
    EXPECT(normpre_default_hparams(nullptr) == NORMPRE_ERR_INVALID_ARG);
    EXPECT(normpre_default_hparams(&hp) == NORMPRE_OK);
    EXPECT(hp.ns_iters == 5 && hp.rank == 32 && hp.oversample == 8 && hp.power_iters == 1);
    EXPECT(std::strlen(normpre_version()) > 0);

    // Validation: valid lists, every error class, message truncation.
    const int64_t ok_shapes[] = {768, 2304, 3072, 768, 1, 300, 300, 1};
    char msg[256];
    for (int variant = 0; variant < 4; ++variant)
        EXPECT(normpre_validate(variant, 4, ok_shapes, &hp, msg, sizeof msg) == NORMPRE_OK);
    EXPECT(normpre_validate(0, 0, nullptr, &hp, msg, sizeof msg) == NORMPRE_OK);
    EXPECT(normpre_validate(0, 1, nullptr, &hp, msg, sizeof msg) == NORMPRE_ERR_INVALID_ARG);
    EXPECT(normpre_validate(0, 1, ok_shapes, nullptr, msg, sizeof msg) == NORMPRE_ERR_INVALID_ARG);
    EXPECT(normpre_validate(9, 1, ok_shapes, &hp, msg, sizeof msg) == NORMPRE_ERR_INVALID_ARG);
    EXPECT(normpre_validate(0, -1, ok_shapes, &hp, msg, sizeof msg) == NORMPRE_ERR_INVALID_ARG);
    const int64_t bad_shape[] = {0, 5};
    EXPECT(normpre_validate(0, 1, bad_shape, &hp, msg, sizeof msg) == NORMPRE_ERR_INVALID_ARG);
    const int64_t huge[] = {int64_t(1) << 21, 4};
    EXPECT(normpre_validate(0, 1, huge, &hp, msg, sizeof msg) == NORMPRE_ERR_UNSUPPORTED);
    const int64_t big_elems[] = {int64_t(1) << 20, int64_t(1) << 12};
    EXPECT(normpre_validate(0, 1, big_elems, &hp, msg, sizeof msg) == NORMPRE_ERR_UNSUPPORTED);
    const int64_t long_rows[] = {8, 40000};
    EXPECT(normpre_validate(0, 1, long_rows, &hp, msg, sizeof msg) == NORMPRE_ERR_UNSUPPORTED);
    char tiny[1] = {'x'};
    EXPECT(normpre_validate(0, 1, bad_shape, &hp, tiny, 1) == NORMPRE_ERR_INVALID_ARG && tiny[0] == '\0');
    EXPECT(normpre_validate(0, 1, bad_shape, &hp, nullptr, 0) == NORMPRE_ERR_INVALID_ARG);
    normpre_hparams h = hp;
    h.lr = NAN;
    EXPECT(normpre_validate(0, 1, ok_shapes, &h, msg, sizeof msg) == NORMPRE_ERR_INVALID_ARG);
    h = hp;
    h.flags = 0xffffffffu;
    EXPECT(normpre_validate(1, 1, ok_shapes, &h, msg, sizeof msg) == NORMPRE_ERR_INVALID_ARG);
    h = hp;
    h.flags = NORMPRE_FLAG_CHECK_FINITE;
    EXPECT(normpre_validate(NORMPRE_VARIANT_MUON, 1, ok_shapes, &h, msg, sizeof msg) == NORMPRE_ERR_INVALID_ARG);
    h = hp;
    h.rank = 400;
    h.oversample = 0;
    const int64_t wide[] = {1000, 1000};
    EXPECT(normpre_validate(1, 1, wide, &h, msg, sizeof msg) == NORMPRE_ERR_UNSUPPORTED);

    // Workspace size (host only): the plan for a whole stack, both variants.
    std::vector<int64_t> stack;
    for (int l = 0; l < 12; ++l) {
        const int64_t per[] = {768, 2304, 768, 768, 768, 3072, 3072, 768};
        stack.insert(stack.end(), per, per + 8);
    }
    int64_t bytes = -1;
    EXPECT(normpre_workspace_size(0, 48, stack.data(), &hp, &bytes) == NORMPRE_OK && bytes > 0);
    int64_t bytes_l = -1;
    EXPECT(normpre_workspace_size(1, 48, stack.data(), &hp, &bytes_l) == NORMPRE_OK && bytes_l > 0);
    h = hp;
    h.flags = NORMPRE_FLAG_CHECK_FINITE;
    int64_t bytes_c = -1;
    EXPECT(normpre_workspace_size(0, 48, stack.data(), &h, &bytes_c) == NORMPRE_OK && bytes_c > bytes);
    EXPECT(normpre_workspace_size(0, 48, stack.data(), &hp, nullptr) == NORMPRE_ERR_INVALID_ARG);
    EXPECT(normpre_workspace_size(0, 1, bad_shape, &hp, &bytes) == NORMPRE_ERR_INVALID_ARG);

    // Energy split (host only).
    const double eigs[] = {9.0, 4.0, 1.0, 0.25, 0.0, -1e-12};
    double out[4];
    EXPECT(normpre_energy_split(eigs, 6, 1, out) == NORMPRE_OK);
    EXPECT(std::fabs(out[0] - 4.0) < 1e-15 && std::fabs(out[1] - 1.0) < 1e-15 && std::fabs(out[2] - 0.25) < 1e-15);
    EXPECT(normpre_energy_split(nullptr, 6, 1, out) == NORMPRE_ERR_INVALID_ARG);
    EXPECT(normpre_energy_split(eigs, -1, 1, out) == NORMPRE_ERR_INVALID_ARG);

    // Entry points given no context: documented error, message available.
    float* p[1] = {nullptr};
    EXPECT(normpre_step(nullptr, 0, 1, p, p, p, ok_shapes, &hp, nullptr) == NORMPRE_ERR_NOT_INITIALIZED);
    EXPECT(normpre_step_noalloc(nullptr, 0, 1, p, p, p, ok_shapes, &hp, nullptr) == NORMPRE_ERR_NOT_INITIALIZED);
    EXPECT(std::strlen(normpre_last_error(nullptr)) > 0);
    EXPECT(normpre_reserve(nullptr, 0, 1, ok_shapes, &hp, nullptr) == NORMPRE_ERR_NOT_INITIALIZED);
    EXPECT(normpre_workspace_bytes(nullptr, &bytes) == NORMPRE_ERR_NOT_INITIALIZED);
    int64_t counts[1];
    EXPECT(normpre_nonfinite_counts(nullptr, counts, 1) == NORMPRE_ERR_NOT_INITIALIZED);
    double cosv[1], mean = 0;
    EXPECT(normpre_descent_alignment(nullptr, 1, nullptr, nullptr, nullptr, ok_shapes, 1.f, 0.f, cosv, &mean,
                                     nullptr) == NORMPRE_ERR_NOT_INITIALIZED);
    EXPECT(normpre_kernel_stats(nullptr, 0, nullptr, nullptr, nullptr, nullptr, nullptr, 0) ==
           NORMPRE_ERR_NOT_INITIALIZED);
    EXPECT(normpre_debug_fetch(nullptr, 0, 0, counts, 8, nullptr) == NORMPRE_ERR_NOT_INITIALIZED);
    EXPECT(normpre_sketch_omega(1, 0, 0, 0, 4, nullptr, nullptr) == NORMPRE_ERR_INVALID_ARG);
    normpre_destroy(nullptr);

    // Context creation: null argument, a device that does not exist.
    EXPECT(normpre_init(nullptr, 0) == NORMPRE_ERR_INVALID_ARG);
    normpre_ctx* ctx = reinterpret_cast<normpre_ctx*>(&hp);
    EXPECT(normpre_init(&ctx, 1 << 20) == NORMPRE_ERR_HIP && ctx == nullptr);

    std::printf("abi host check: %d failure(s)\n", failures);
    return failures;
}
