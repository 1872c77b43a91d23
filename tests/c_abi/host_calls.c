/* The C ABI from plain C99 (no GPU): plan creation and introspection,
 * custom plans, GenModel terms and selection, error reporting.  Prints one
 * line per check and exits non-zero on the first failure.  Built and run by
 * tests/test_c_abi_host.py. */
#include <stdio.h>
#include <stdint.h>
#include <string.h>

#include "ar_plan.h"

static int failures = 0;
#define CHECK(cond, what)                                                  \
    do {                                                                   \
        if (cond) {                                                        \
            printf("ok   %s\n", what);                                     \
        } else {                                                           \
            printf("FAIL %s (%s)\n", what, ar_last_error());               \
            ++failures;                                                    \
        }                                                                  \
    } while (0)

int main(void) {
    /* tree (8, 8) over 64 processors: 2 ReduceScatter + 2 AllGather phases */
    const int32_t fan[2] = {8, 8};
    ar_topology topo = {AR_TREE, 2, fan};
    ar_plan* plan = NULL;
    CHECK(ar_plan_create(64, 1 << 16, AR_F32, &topo, &plan) == AR_OK && plan, "create tree (8, 8)");
    int32_t n = 0, dtype = -1, phases = 0;
    int64_t N = 0, steps = 0;
    CHECK(ar_plan_info(plan, &n, &N, &dtype, &phases, &steps) == AR_OK && n == 64 &&
              N == (1 << 16) && dtype == AR_F32 && phases == 4,
          "info");
    /* level-0 reduce: 64 steps of 8 sources over N / 8 elements each */
    int32_t op = -1;
    int64_t first = -1, count = 0, bytes = 0;
    CHECK(ar_plan_phase_info(plan, 0, &op, &first, &count, &bytes) == AR_OK && op == AR_OP_REDUCE &&
              first == 0 && count == 64 && bytes == 64LL * 9 * ((1 << 16) / 8) * 4,
          "phase 0: 64 eight-way reduces, (k + 1) * len * e bytes each");
    ar_step st;
    CHECK(ar_plan_get_step(plan, 0, &st) == AR_OK && st.nsrc == 8 && st.op == AR_OP_REDUCE, "step 0");
    int64_t red = 0, cpy = 0;
    CHECK(ar_plan_bytes(plan, &red, &cpy) == AR_OK && red > 0 && cpy > 0, "plan bytes");
    int64_t b = -1, e = -1;
    CHECK(ar_plan_owner(plan, 9, &b, &e) == AR_OK && e - b == (1 << 16) / 64, "owner of processor 9");
    int32_t launches = 0;
    CHECK(ar_plan_num_launches(plan, &launches) == AR_OK && launches >= 1, "launches");
    int32_t kernel = -1;
    CHECK(ar_plan_launch_kernel(plan, 0, &kernel) == AR_OK && kernel >= AR_KERNEL_PHASE &&
              kernel <= AR_KERNEL_STREAM,
          "kernel of launch 0");
    CHECK(ar_plan_launch_kernel(plan, launches, &kernel) == AR_ERR_INVALID_ARG,
          "launch index out of range refused");
    double terms[AR_GENMODEL_TERMS];
    CHECK(ar_genmodel_terms(plan, (int64_t)256 << 20, terms) == AR_OK && terms[0] == 4.0 &&
              terms[1] == 8 + 8 + 1 + 1 && terms[2] + terms[3] == (double)red,
          "GenModel terms");
    const int64_t tiers[2] = {(int64_t)256 << 20, (int64_t)32 << 20};
    double tiered[4 + 2 * 2];
    CHECK(ar_genmodel_terms_tiered(plan, 2, tiers, tiered) == AR_OK && tiered[0] == 4.0 &&
              tiered[2] + tiered[3] + tiered[4] == (double)red,
          "GenModel tiered terms");
    CHECK(ar_genmodel_terms_tiered(plan, 0, tiers, tiered) == AR_ERR_INVALID_ARG,
          "no tier refused");
    CHECK(ar_plan_destroy(plan) == AR_OK, "destroy");
    CHECK(ar_plan_destroy(NULL) == AR_OK, "destroy NULL");

    /* a custom plan: phase 0 reduces [0, 8) of 0 and 1 into 0, phase 1
     * copies it to 1 */
    const int32_t s01[2] = {0, 1}, s0[1] = {0};
    ar_step cs[2] = {{0, AR_OP_REDUCE, 0, 2, s01, 0, 8}, {1, AR_OP_COPY, 1, 1, s0, 0, 8}};
    CHECK(ar_plan_create_custom(2, 8, AR_BF16, cs, 2, &plan) == AR_OK, "custom plan");
    ar_plan_destroy(plan);
    /* a hazard: the copy writes what the reduce of the same phase reads */
    cs[1].phase = 0;
    plan = (ar_plan*)&cs;  /* must be reset to NULL on failure */
    CHECK(ar_plan_create_custom(2, 8, AR_BF16, cs, 2, &plan) == AR_ERR_INVALID_ARG && plan == NULL,
          "hazard refused, out set to NULL");

    /* GenTree on the 6-server tree [3 servers, 2 servers] */
    const int32_t tree[6] = {2, 3, 0, 0, 0, 2};
    const int32_t tree_ok[8] = {2, 3, 0, 0, 0, 2, 0, 0};
    CHECK(ar_plan_create_gentree(100, AR_F32, 6, tree, &plan) == AR_ERR_INVALID_ARG, "malformed tree");
    CHECK(ar_plan_create_gentree(100, AR_F32, 8, tree_ok, &plan) == AR_OK, "GenTree plan");
    CHECK(ar_plan_info(plan, &n, NULL, NULL, NULL, NULL) == AR_OK && n == 5, "five servers");
    ar_plan_destroy(plan);

    /* GenModel selection: with only a per-round cost, co-located PS (two
     * rounds) wins */
    const double rounds_only[AR_GENMODEL_TERMS] = {1.0, 0, 0, 0, 0, 0};
    int32_t kind = -1, levels = -1, fanin[3];
    double sec = 0;
    CHECK(ar_genmodel_select(16, 1 << 20, AR_F32, rounds_only, 0, 3, &kind, &levels, fanin, &sec) ==
                  AR_OK && kind == AR_CPS && levels == 0 && sec == 2.0,
          "GenModel picks co-located PS on rounds alone");
    const double rounds_only8[4 + 2 * 2] = {1.0, 0, 0, 0, 0, 0, 0, 0};
    CHECK(ar_genmodel_select_tiered(16, 1 << 20, AR_F32, rounds_only8, 2, tiers, 3, &kind, &levels,
                                    fanin, &sec) == AR_OK && kind == AR_CPS && sec == 2.0,
          "tiered GenModel picks co-located PS on rounds alone");

    /* errors */
    CHECK(ar_plan_create(0, 10, AR_F32, &topo, &plan) == AR_ERR_INVALID_ARG, "n = 0 refused");
    CHECK(strlen(ar_last_error()) > 0, "error text");
    CHECK(strcmp(ar_status_string(AR_ERR_UNSUPPORTED), "") != 0, "status string");
    ar_timer* t = NULL;
    CHECK(ar_timer_create(4, &t) == AR_OK && ar_timer_destroy(t) == AR_OK, "timer");
    printf("%d failures\n", failures);
    return failures != 0;
}
