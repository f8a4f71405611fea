/*
 * Host-side argument checks of the C ABI (include/olive_score.h), run under
 * AddressSanitizer and UndefinedBehaviorSanitizer on a machine without a GPU.
 *
 * Every call here must return before it reaches the device: malformed descriptors,
 * NULL pointers and NULL contexts are rejected on the host with the documented
 * status. A descriptor that passes every host check makes init ask the HIP runtime
 * for a device; without one it must fail with OLIVE_E_HIP and release its partly
 * built context cleanly. The sanitizers abort on any invalid memory access or
 * undefined behaviour along these paths. Prints "ok <n>" and exits 0 when every
 * check holds.
 */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "olive_score.h"

static int n_checks = 0, n_failed = 0;

#define CHECK(cond)                                                              \
    do {                                                                         \
        ++n_checks;                                                              \
        if (!(cond)) {                                                           \
            ++n_failed;                                                          \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
        }                                                                        \
    } while (0)

static olive_score_desc good_desc(void) {
    olive_score_desc d;
    memset(&d, 0, sizeof(d));
    d.vocab = 1000;
    d.d_student = 64;
    d.d_teacher = 96;
    d.dtype = OLIVE_BF16;
    d.w_layout = OLIVE_W_DV;
    d.logit_scale_student = 1.0f;
    d.logit_scale_teacher = 1.0f;
    d.max_positions = 64;
    d.max_seqs = 2;
    d.flags = 0;
    return d;
}

/* Non-NULL stand-ins for device pointers: never dereferenced on the host paths. */
static char dev_w[64];

static olive_status init_with(const olive_score_desc *d) {
    olive_score_ctx *ctx = (olive_score_ctx *)&n_checks;   /* must be overwritten */
    olive_status s = olive_score_init(&ctx, d, dev_w, dev_w, NULL);
    CHECK(ctx == NULL);
    return s;
}

int main(void) {
    /* status strings: every code, and an unknown one */
    for (int c = OLIVE_OK; c <= OLIVE_E_LIMIT; ++c) {
        const char *s = olive_status_string((olive_status)c);
        CHECK(s != NULL && strncmp(s, "OLIVE_", 6) == 0);
    }
    CHECK(strstr(olive_status_string((olive_status)99), "unknown") != NULL);
    CHECK(strstr(olive_status_string((olive_status)-5), "unknown") != NULL);

    /* init: NULL arguments */
    olive_score_desc d = good_desc();
    olive_score_ctx *ctx = NULL;
    CHECK(olive_score_init(NULL, &d, dev_w, dev_w, NULL) == OLIVE_E_NULL);
    CHECK(olive_score_init(&ctx, NULL, dev_w, dev_w, NULL) == OLIVE_E_NULL);
    CHECK(olive_score_init(&ctx, &d, NULL, dev_w, NULL) == OLIVE_E_NULL && ctx == NULL);
    CHECK(olive_score_init(&ctx, &d, dev_w, NULL, NULL) == OLIVE_E_NULL && ctx == NULL);

    /* init: every malformed descriptor field */
    d = good_desc(); d.dtype = 7;                     CHECK(init_with(&d) == OLIVE_E_DTYPE);
    d = good_desc(); d.w_layout = 5;                  CHECK(init_with(&d) == OLIVE_E_DTYPE);
    d = good_desc(); d.vocab = 0;                     CHECK(init_with(&d) == OLIVE_E_SHAPE);
    d = good_desc(); d.vocab = (int64_t)1 << 31;      CHECK(init_with(&d) == OLIVE_E_SHAPE);
    d = good_desc(); d.vocab = -3;                    CHECK(init_with(&d) == OLIVE_E_SHAPE);
    d = good_desc(); d.d_student = 0;                 CHECK(init_with(&d) == OLIVE_E_SHAPE);
    d = good_desc(); d.d_teacher = -1;                CHECK(init_with(&d) == OLIVE_E_SHAPE);
    d = good_desc(); d.max_positions = 0;             CHECK(init_with(&d) == OLIVE_E_SHAPE);
    d = good_desc(); d.max_positions = (int64_t)1 << 40; CHECK(init_with(&d) == OLIVE_E_SHAPE);
    d = good_desc(); d.max_seqs = 0;                  CHECK(init_with(&d) == OLIVE_E_SHAPE);
    d = good_desc(); d.d_student = 12289;             CHECK(init_with(&d) == OLIVE_E_UNSUPPORTED);
    d = good_desc(); d.d_teacher = 1 << 30;           CHECK(init_with(&d) == OLIVE_E_UNSUPPORTED);
    d = good_desc(); d.logit_scale_student = 0.0f;    CHECK(init_with(&d) == OLIVE_E_RANGE);
    d = good_desc(); d.logit_scale_student = INFINITY; CHECK(init_with(&d) == OLIVE_E_RANGE);
    d = good_desc(); d.logit_scale_teacher = -1.0f;   CHECK(init_with(&d) == OLIVE_E_RANGE);
    d = good_desc(); d.logit_scale_teacher = NAN;     CHECK(init_with(&d) == OLIVE_E_RANGE);
    d = good_desc(); d.flags = 64;                    CHECK(init_with(&d) == OLIVE_E_RANGE);
    d = good_desc(); d.flags = -1;                    CHECK(init_with(&d) == OLIVE_E_RANGE);

    /* a descriptor that passes the host checks: without a device, init fails in the
       HIP runtime and frees what it built */
    d = good_desc();
    CHECK(init_with(&d) == OLIVE_E_HIP);
    d = good_desc(); d.d_teacher = 0; d.flags = OLIVE_FLAG_TOPK | OLIVE_FLAG_BACKWARD;
    {
        olive_status s = init_with(&d);
        CHECK(s == OLIVE_E_HIP || s == OLIVE_E_UNSUPPORTED);
    }

    /* every call on a NULL context */
    olive_batch b;
    memset(&b, 0, sizeof(b));
    olive_score_outputs o;
    memset(&o, 0, sizeof(o));
    o.size = (int32_t)sizeof(o);
    olive_spans sp;
    memset(&sp, 0, sizeof(sp));
    sp.size = (int32_t)sizeof(sp);
    olive_grad_outputs g;
    memset(&g, 0, sizeof(g));
    g.size = (int32_t)sizeof(g);
    float f[4];
    int32_t code = 0;
    int64_t stats[6];
    CHECK(olive_token_logprobs(NULL, &b, f, NULL, NULL, NULL, NULL) == OLIVE_E_NULL);
    CHECK(olive_kl_masked(NULL, &b, f, NULL, NULL, NULL, NULL, NULL, NULL, NULL) == OLIVE_E_NULL);
    CHECK(olive_score_batch(NULL, &b, &o, NULL) == OLIVE_E_NULL);
    CHECK(olive_score_batch_spans(NULL, &b, &sp, &o, NULL) == OLIVE_E_NULL);
    CHECK(olive_score_backward(NULL, &b, NULL, &g, NULL) == OLIVE_E_NULL);
    CHECK(olive_score_last_error(NULL, &code) == OLIVE_E_NULL);
    CHECK(olive_score_last_stats(NULL, stats) == OLIVE_E_NULL);
    CHECK(olive_score_kernel_times(NULL, f, 1) == OLIVE_E_NULL);
    CHECK(olive_score_free(NULL) == OLIVE_OK);

    /* the no-allocation entry point: host checks before any device call */
    d = good_desc();
    d.w_layout = OLIVE_W_VD;
    CHECK(olive_kl_masked_static(NULL, dev_w, dev_w, &b, f, NULL, NULL, NULL, NULL, NULL, NULL,
                                 NULL) == OLIVE_E_NULL);
    CHECK(olive_kl_masked_static(&d, dev_w, dev_w, &b, NULL, NULL, NULL, NULL, NULL, NULL, NULL,
                                 NULL) == OLIVE_E_NULL);
    CHECK(olive_kl_masked_static(&d, NULL, dev_w, &b, f, NULL, NULL, NULL, NULL, NULL, NULL,
                                 NULL) == OLIVE_E_NULL);
    {
        olive_score_desc e = d; e.w_layout = OLIVE_W_DV;
        CHECK(olive_kl_masked_static(&e, dev_w, dev_w, &b, f, NULL, NULL, NULL, NULL, NULL, NULL,
                                     NULL) == OLIVE_E_UNSUPPORTED);
        e = d; e.flags = OLIVE_FLAG_KERNEL_TIMING;
        CHECK(olive_kl_masked_static(&e, dev_w, dev_w, &b, f, NULL, NULL, NULL, NULL, NULL, NULL,
                                     NULL) == OLIVE_E_UNSUPPORTED);
        e = d; e.d_teacher = 0;
        CHECK(olive_kl_masked_static(&e, dev_w, dev_w, &b, f, NULL, NULL, NULL, NULL, NULL, NULL,
                                     NULL) == OLIVE_E_UNSUPPORTED);
        e = d; e.max_positions = 8193;
        CHECK(olive_kl_masked_static(&e, dev_w, dev_w, &b, f, NULL, NULL, NULL, NULL, NULL, NULL,
                                     NULL) == OLIVE_E_LIMIT);
        e = d; e.vocab = 262145;
        CHECK(olive_kl_masked_static(&e, dev_w, dev_w, &b, f, NULL, NULL, NULL, NULL, NULL, NULL,
                                     NULL) == OLIVE_E_LIMIT);
        e = d; e.max_seqs = 257;
        CHECK(olive_kl_masked_static(&e, dev_w, dev_w, &b, f, NULL, NULL, NULL, NULL, NULL, NULL,
                                     NULL) == OLIVE_E_LIMIT);
        e = d; e.dtype = 9;
        CHECK(olive_kl_masked_static(&e, dev_w, dev_w, &b, f, NULL, NULL, NULL, NULL, NULL, NULL,
                                     NULL) == OLIVE_E_DTYPE);
    }
    /* within every limit: without a device the call fails in the HIP runtime */
    CHECK(olive_kl_masked_static(&d, dev_w, dev_w, &b, f, NULL, NULL, NULL, NULL, NULL, NULL,
                                 NULL) == OLIVE_E_HIP);

    if (n_failed) {
        fprintf(stderr, "%d of %d checks failed\n", n_failed, n_checks);
        return 1;
    }
    printf("ok %d\n", n_checks);
    return 0;
}
