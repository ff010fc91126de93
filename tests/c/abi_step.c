/* A plain C client of the library's ABI (include/fc.h), with no Python and
 * no torch: it allocates device buffers with the HIP runtime's C API, runs
 * one fc_step, fc_plan_balance, fc_tree_reduce, fc_sgd_step on that sum and
 * fc_broadcast of w' per schedule on a small ragged segment table, and
 * compares every element bit for bit with the oracle's C functions (the
 * oracle is linked as test infrastructure) on the same inputs.  Exit status
 * 0 when everything matches; each failure is printed. */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "fc.h"

/* the oracle's entry points (oracle/fc_oracle.c) */
typedef struct {
    uint64_t offset, length;
    float lr_mult, decay_mult;
} orc_segment;
int orc_tree_reduce(const orc_segment* segs, int nseg, int K, int dtype, int order, const void* const* grads,
                    float* out);
int orc_step(const orc_segment* segs, int nseg, int K, int dtype, int order, const void* const* grads, float* w,
             float* v, float lr, float mu, float wd, int batch, float* scratch, float* out, float* const* bcast_dst);
int orc_broadcast(const orc_segment* segs, int nseg, int K, const float* src, float* const* dst);

enum { K = 37, NSEG = 3, N = 5248 };

static uint32_t state = 12345u;
static float draw(float scale) {
    state = state * 1664525u + 1013904223u; /* a linear congruential generator */
    return ((float)(state >> 8) / 16777216.0f - 0.5f) * scale;
}

#define HIP_OK(x)                                                        \
    do {                                                                 \
        if ((x) != hipSuccess) {                                         \
            fprintf(stderr, "c client: %s failed at line %d\n", #x, __LINE__); \
            exit(2);                                                     \
        }                                                                \
    } while (0)

static int compare(const char* what, int schedule, const float* got, const float* want, size_t n) {
    size_t bad = 0;
    for (size_t i = 0; i < n; ++i)
        if (memcmp(&got[i], &want[i], sizeof(float)) != 0) ++bad;
    if (bad) fprintf(stderr, "c client: schedule %d: %s differs from the oracle in %zu elements\n", schedule, what, bad);
    return bad != 0;
}

int main(void) {
    const fc_segment segs[NSEG] = {{0, 1000, 1.0f, 1.0f}, {1024, 4097, 2.0f, 0.0f}, {5184, 3, 1.0f, 1.0f}};
    orc_segment osegs[NSEG];
    for (int j = 0; j < NSEG; ++j) {
        osegs[j].offset = segs[j].offset;
        osegs[j].length = segs[j].length;
        osegs[j].lr_mult = segs[j].lr_mult;
        osegs[j].decay_mult = segs[j].decay_mult;
    }
    const float lr = 0.01f, mu = 0.9f, wd = 5e-4f;
    const int batch = 256;

    float* reps = malloc(sizeof(float) * K * N);
    float* w0 = malloc(sizeof(float) * N);
    float* v0 = malloc(sizeof(float) * N);
    float* w = malloc(sizeof(float) * N);
    float* v = malloc(sizeof(float) * N);
    float* out = malloc(sizeof(float) * N);
    float* scratch = malloc(sizeof(float) * N);
    float* got = malloc(sizeof(float) * N);
    float* fill = malloc(sizeof(float) * N);
    float* bc = malloc(sizeof(float) * K * N);
    const void* host_rows[K];
    float* bc_rows[K];
    if (!reps || !w0 || !v0 || !w || !v || !out || !scratch || !got || !fill || !bc) return 2;
    for (int i = 0; i < N; ++i) fill[i] = -2.0f;  /* what the broadcast must leave outside the segments */
    for (int i = 0; i < K * N; ++i) reps[i] = draw(0.01f);
    for (int i = 0; i < N; ++i) {
        w0[i] = draw(0.1f);
        v0[i] = draw(0.001f);
    }
    for (int k = 0; k < K; ++k) host_rows[k] = reps + (size_t)k * N;

    float *d_reps, *d_w, *d_v, *d_out, *d_w2, *d_v2, *d_bc;
    HIP_OK(hipMalloc((void**)&d_reps, sizeof(float) * K * N));
    HIP_OK(hipMalloc((void**)&d_w, sizeof(float) * N));
    HIP_OK(hipMalloc((void**)&d_v, sizeof(float) * N));
    HIP_OK(hipMalloc((void**)&d_out, sizeof(float) * N));
    HIP_OK(hipMalloc((void**)&d_w2, sizeof(float) * N));
    HIP_OK(hipMalloc((void**)&d_v2, sizeof(float) * N));
    HIP_OK(hipMalloc((void**)&d_bc, sizeof(float) * K * N));
    float* dev_bc[K];
    for (int k = 0; k < K; ++k) {
        dev_bc[k] = d_bc + (size_t)k * N;
        bc_rows[k] = bc + (size_t)k * N;
    }
    HIP_OK(hipMemcpy(d_reps, reps, sizeof(float) * K * N, hipMemcpyHostToDevice));
    const void* dev_rows[K];
    for (int k = 0; k < K; ++k) dev_rows[k] = d_reps + (size_t)k * N;

    /* errors are codes, never aborts */
    fc_plan* none = NULL;
    if (fc_plan_create(&none, segs, NSEG, 0, FC_F32, FC_ORDER_TREE) != FC_EINVAL || none != NULL ||
        fc_strerror(FC_EINVAL) == NULL) {
        fprintf(stderr, "c client: an invalid plan was not refused\n");
        return 1;
    }

    int failed = 0;
    const int schedules[5] = {FC_SCHED_AUTO, FC_SCHED_FUSED, FC_SCHED_TWO_PASS, FC_SCHED_RESIDENT,
                              FC_SCHED_RESIDENT_ONE_LAUNCH};
    for (int si = 0; si < 5; ++si) {
        fc_launch_opts opts;
        memset(&opts, 0, sizeof opts);
        opts.schedule = schedules[si];
        fc_plan* plan = NULL;
        int rc = fc_plan_create_ex(&plan, segs, NSEG, K, FC_F32, FC_ORDER_TREE, &opts);
        if (rc != FC_OK) {
            fprintf(stderr, "c client: fc_plan_create_ex: %s\n", fc_strerror(rc));
            return 1;
        }
        fc_plan_info info;
        if (fc_plan_query(plan, &info) != FC_OK ||
            (schedules[si] != FC_SCHED_AUTO && info.schedule != schedules[si])) {
            fprintf(stderr, "c client: schedule %d: the plan reports schedule %d\n", schedules[si], info.schedule);
            return 1;
        }
        /* one fused step on the device and in the oracle, same inputs */
        HIP_OK(hipMemcpy(d_w, w0, sizeof(float) * N, hipMemcpyHostToDevice));
        HIP_OK(hipMemcpy(d_v, v0, sizeof(float) * N, hipMemcpyHostToDevice));
        rc = fc_step(plan, dev_rows, d_w, d_v, lr, mu, wd, batch, NULL, NULL, NULL);
        /* XCD-aware shares from the step's record (resident plans; a no-op
           for the others): the reduce that follows runs on the new shares */
        float rates[16];
        if (rc == FC_OK) rc = fc_plan_balance(plan, NULL, rates, 16);
        if (rc == FC_OK) rc = fc_tree_reduce(plan, dev_rows, d_out, NULL);
        /* the composed path: SGD from that raw sum, then w' to K copies */
        HIP_OK(hipMemcpy(d_w2, w0, sizeof(float) * N, hipMemcpyHostToDevice));
        HIP_OK(hipMemcpy(d_v2, v0, sizeof(float) * N, hipMemcpyHostToDevice));
        for (int k = 0; k < K; ++k) HIP_OK(hipMemcpy(dev_bc[k], fill, sizeof(float) * N, hipMemcpyHostToDevice));
        if (rc == FC_OK) rc = fc_sgd_step(plan, d_w2, d_v2, d_out, lr, mu, wd, batch, NULL);
        if (rc == FC_OK) rc = fc_broadcast(plan, d_w2, dev_bc, NULL);
        if (rc != FC_OK) {
            fprintf(stderr, "c client: schedule %d: %s\n", schedules[si], fc_strerror(rc));
            return 1;
        }
        HIP_OK(hipDeviceSynchronize());
        memcpy(w, w0, sizeof(float) * N);
        memcpy(v, v0, sizeof(float) * N);
        memcpy(out, w0, sizeof(float) * N);  /* gaps keep whatever the buffer held */
        memcpy(scratch, w0, sizeof(float) * N);
        if (orc_step(osegs, NSEG, K, 0, 0, host_rows, w, v, lr, mu, wd, batch, scratch, NULL, NULL) != 0) return 2;
        HIP_OK(hipMemcpy(got, d_w, sizeof(float) * N, hipMemcpyDeviceToHost));
        failed |= compare("w'", schedules[si], got, w, N);
        HIP_OK(hipMemcpy(got, d_v, sizeof(float) * N, hipMemcpyDeviceToHost));
        failed |= compare("v'", schedules[si], got, v, N);
        if (orc_tree_reduce(osegs, NSEG, K, 0, 0, host_rows, out) != 0) return 2;
        HIP_OK(hipMemcpy(got, d_out, sizeof(float) * N, hipMemcpyDeviceToHost));
        for (int j = 0; j < NSEG; ++j)  /* only segment elements are defined in d_out */
            failed |= compare("raw sum", schedules[si], got + segs[j].offset, out + segs[j].offset,
                              (size_t)segs[j].length);
        HIP_OK(hipMemcpy(got, d_w2, sizeof(float) * N, hipMemcpyDeviceToHost));
        failed |= compare("w' (composed)", schedules[si], got, w, N);
        HIP_OK(hipMemcpy(got, d_v2, sizeof(float) * N, hipMemcpyDeviceToHost));
        failed |= compare("v' (composed)", schedules[si], got, v, N);
        for (int k = 0; k < K; ++k) memcpy(bc_rows[k], fill, sizeof(float) * N);
        if (orc_broadcast(osegs, NSEG, K, w, bc_rows) != 0) return 2;
        for (int k = 0; k < K; ++k) {
            HIP_OK(hipMemcpy(got, dev_bc[k], sizeof(float) * N, hipMemcpyDeviceToHost));
            failed |= compare("broadcast copy", schedules[si], got, bc_rows[k], N);
        }
        fc_plan_destroy(plan);
    }
    hipFree(d_reps);
    hipFree(d_w);
    hipFree(d_v);
    hipFree(d_out);
    hipFree(d_w2);
    hipFree(d_v2);
    hipFree(d_bc);
    free(reps), free(w0), free(v0), free(w), free(v), free(out), free(scratch), free(got), free(fill), free(bc);
    if (!failed)
        printf("c client: fc_step, fc_tree_reduce, fc_sgd_step and fc_broadcast bit-exact vs the oracle "
               "(K=%d, %d segments, 4 schedules)\n", K, NSEG);
    return failed;
}
