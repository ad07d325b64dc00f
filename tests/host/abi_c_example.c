/* The C ABI from plain C99: plan a batch with pp_plan_bounds and pp_pack (host code, no GPU
 * needed) and print its rows, segments and restart positions.  Built and run by
 * tests/test_abi_c.py with gcc -std=c99 -pedantic -Werror against libprepack.so; also a
 * starting point for C callers (a GPU program continues with pp_prefill_workspace_size and
 * pp_prefill on device copies of the plan arrays). */
#include <stdio.h>
#include <stdlib.h>

#include "prepack.h"

static int32_t* alloc_i32(int64_t n) { return (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t)); }

int main(void) {
    const int32_t lengths[6] = {5, 3, 8, 2, 6, 1};   /* section 3.1: FFD into rows of 8 */
    const int32_t k = 6, capacity = 8;
    int64_t slot_cap = 0, qtile_cap = 0, mtile_cap = 0;
    pp_plan plan;
    pp_status st;
    int32_t r, s, t, real = 0;

    printf("library %s\n", pp_version());
    st = pp_plan_bounds(k, capacity, &slot_cap, &qtile_cap, &mtile_cap);
    if (st != PP_OK) {
        fprintf(stderr, "pp_plan_bounds: %s\n", pp_last_error());
        return 1;
    }
    plan.slot_cap = slot_cap;
    plan.qtile_cap = qtile_cap;
    plan.mtile_cap = mtile_cap;
    plan.row_seg_ptr = alloc_i32(k + 1);
    plan.seg_prompt = alloc_i32(k);
    plan.seg_start = alloc_i32(k);
    plan.seg_len = alloc_i32(k);
    plan.prompt_kv_off = alloc_i32(k + 1);
    plan.slot_seg = alloc_i32(slot_cap);
    plan.slot_pos = alloc_i32(slot_cap);
    plan.slot_kv = alloc_i32(slot_cap);
    plan.qtile_seg = alloc_i32(qtile_cap);
    plan.qtile_q0 = alloc_i32(qtile_cap);
    plan.mtile_m0 = alloc_i32(mtile_cap);

    st = pp_pack(lengths, k, capacity, &plan);
    if (st != PP_OK) {
        fprintf(stderr, "pp_pack: %s\n", pp_last_error());
        return 1;
    }
    printf("%d prompts, %d tokens, %d rows of %d\n", plan.k, plan.total_len, plan.n_rows, plan.capacity);
    for (r = 0; r < plan.n_rows; ++r) {
        printf("row %d:", r);
        for (s = plan.row_seg_ptr[r]; s < plan.row_seg_ptr[r + 1]; ++s)
            printf(" prompt %d (len %d)", plan.seg_prompt[s], plan.seg_len[s]);
        printf(" | positions");
        for (t = 0; t < plan.capacity; ++t) {
            const int64_t slot = (int64_t)r * plan.capacity + t;
            if (plan.slot_seg[slot] < 0) printf(" .");
            else printf(" %d", plan.slot_pos[slot]);
            if (plan.slot_kv[slot] >= 0) ++real;
        }
        printf("\n");
    }
    /* FFD of {8, 6, 5, 3, 2, 1} into rows of 8: [8], [6, 2], [5, 3], [1] */
    if (plan.n_rows != 4 || real != plan.total_len || plan.total_len != 25) {
        fprintf(stderr, "unexpected plan: %d rows, %d real slots\n", plan.n_rows, real);
        return 1;
    }
    /* an invalid call reports its reason */
    if (pp_pack(lengths, k, 4, &plan) != PP_ERR_TOO_LONG) return 1;
    printf("capacity 4: %s\n", pp_last_error());
    free(plan.row_seg_ptr);
    free(plan.seg_prompt);
    free(plan.seg_start);
    free(plan.seg_len);
    free(plan.prompt_kv_off);
    free(plan.slot_seg);
    free(plan.slot_pos);
    free(plan.slot_kv);
    free(plan.qtile_seg);
    free(plan.qtile_q0);
    free(plan.mtile_m0);
    return 0;
}
