/* A plain C program against include/edkm.h: it compiles with gcc (no hipcc,
 * no platform define on the command line), links libedkm.so and checks the
 * host-side argument and call-order errors of the real ABI.  It makes no call
 * that reaches the GPU.  Prints "ok" and exits 0 when every check holds. */
#include <stdio.h>
#include <string.h>

#include "edkm.h"

static int failures = 0;
#define CHECK(cond) do { if (!(cond)) { printf("FAIL line %d: %s\n", __LINE__, #cond); ++failures; } } while (0)

int main(void)
{
    const uint64_t n = 4096;
    const size_t ws = edkm_workspace_bytes(n, 3, 5);
    CHECK(ws > 0 && ws % 256 == 0);
    CHECK(edkm_workspace_bytes(0, 3, 5) == 0);
    CHECK(edkm_workspace_bytes(n, 5, 5) == 0);
    CHECK(edkm_workspace_bytes(n, 3, EDKM_MAX_ITER + 1) == 0);
    CHECK(edkm_workspace_bytes(EDKM_MAX_N + 1ull, 3, 5) == 0);

    /* never dereferenced: every call below is refused on the host */
    void* fake_ws = (void*)((uintptr_t)1 << 40);
    const uint16_t* keys = (const uint16_t*)((uintptr_t)1 << 41);
    float* f = (float*)((uintptr_t)1 << 42);

    edkm_plan plan;
    CHECK(edkm_plan_init(NULL, n, 3, 5, fake_ws, ws) == EDKM_ERR_ARG);
    CHECK(edkm_plan_init(&plan, n, 3, 5, NULL, ws) == EDKM_ERR_WORKSPACE);
    CHECK(edkm_plan_init(&plan, n, 3, 5, fake_ws, ws - 1) == EDKM_ERR_WORKSPACE);
    CHECK(edkm_plan_init(&plan, n, 3, 5, (char*)fake_ws + 16, ws) == EDKM_ERR_WORKSPACE);
    CHECK(edkm_plan_init_ex(&plan, n, 3, 5, 7, fake_ws, ws) == EDKM_ERR_ARG);
    CHECK(edkm_plan_init(&plan, n, 3, 5, fake_ws, ws) == EDKM_OK);

    /* out of order: forward / backward before init_unique */
    CHECK(edkm_forward(&plan, keys, 2e-3f, 0.0f, f, f, f, 0, NULL, NULL) == EDKM_ERR_STATE);
    CHECK(edkm_backward(&plan, keys, f, f, f, NULL) == EDKM_ERR_STATE);
    CHECK(edkm_backward_dense(&plan, keys, f, f, f, NULL) == EDKM_ERR_STATE);
    CHECK(edkm_backward_ex(&plan, keys, f, f, f, EDKM_GRAD_IN_HALF | EDKM_GRAD_OUT_HALF, NULL) == EDKM_ERR_STATE);
    CHECK(edkm_unique_inverse(&plan, keys, (uint16_t*)f, NULL, NULL) == EDKM_ERR_STATE);
    /* bad arguments */
    CHECK(edkm_forward(&plan, keys, 0.0f, 0.0f, f, f, f, 0, NULL, NULL) == EDKM_ERR_ARG);
    CHECK(edkm_forward(&plan, keys, 2e-3f, -1.0f, f, f, f, 0, NULL, NULL) == EDKM_ERR_ARG);
    CHECK(edkm_forward(&plan, keys, 2e-3f, 0.0f, NULL, f, f, 0, NULL, NULL) == EDKM_ERR_ARG);
    CHECK(edkm_init_unique(&plan, NULL, NULL, NULL, 0, NULL) == EDKM_ERR_ARG);
    CHECK(edkm_init_unique(&plan, keys, NULL, NULL, 2, NULL) == EDKM_ERR_ARG);
    CHECK(edkm_palettize(&plan, keys, NULL, (uint8_t*)f, NULL) == EDKM_ERR_ARG);
    CHECK(edkm_plan_set_keyed_mode(&plan, 5) == EDKM_ERR_ARG);
    CHECK(edkm_backward_ex(&plan, keys, f, f, f, 4, NULL) == EDKM_ERR_ARG);   /* unknown flag */
    CHECK(edkm_plan_set_pass_events(&plan, 99, NULL, NULL) == EDKM_ERR_ARG);

    /* a copied record is refused; the original still works */
    edkm_plan copy;
    memcpy(&copy, &plan, sizeof(plan));
    CHECK(edkm_forward(&copy, keys, 2e-3f, 0.0f, f, f, f, 0, NULL, NULL) == EDKM_ERR_ARG);
    CHECK(edkm_plan_set_keyed_mode(&copy, EDKM_KEYED_AUTO) == EDKM_ERR_ARG);
    CHECK(edkm_plan_set_keyed_mode(&plan, EDKM_KEYED_AUTO) == EDKM_OK);

    int code = -1;
    const char* step = NULL;
    const char* msg = NULL;
    CHECK(edkm_plan_hip_error(&plan, &code, &step, &msg) == EDKM_OK && code == 0);
    CHECK(strcmp(edkm_status_str(EDKM_ERR_STATE), "ok") != 0);
    CHECK(strcmp(edkm_status_str(EDKM_OK), "ok") == 0);

    if (failures) return 1;
    printf("ok\n");
    return 0;
}
