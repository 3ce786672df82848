/* A plain C program using libconduit through include/conduit.h only: create a
 * buffer, ingest rows, read the ring state back, sample with a fused gather,
 * check every gathered row against the bytes ingested into the sampled slot,
 * update priorities, take a checkpoint and restore it into a second buffer.
 * Built by __graft_entry__.build() (gcc, C11); run by test_gpu_c_consumer.py.
 * Prints "c consumer ok" and exits 0, or names the failed check and exits 1. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "conduit.h"

#define CHECK(cond, what)                                                   \
    do {                                                                    \
        if (!(cond)) {                                                      \
            fprintf(stderr, "c consumer: %s failed (%s)\n", what, conduit_last_error()); \
            return 1;                                                       \
        }                                                                   \
    } while (0)

enum { CAP = 1000, ROW = 16, N = 600, BATCH = 64 };

static uint64_t splitmix(uint64_t* s) {
    uint64_t z = (*s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static void* dev_copy(const void* h, size_t n) {
    void* d = NULL;
    if (hipMalloc(&d, n) != hipSuccess) return NULL;
    if (hipMemcpy(d, h, n, hipMemcpyHostToDevice) != hipSuccess) return NULL;
    return d;
}

int main(void) {
    static uint8_t obs[N * ROW];
    static int32_t action[N], step[N];
    static float reward[N];
    static uint8_t done[N];
    static uint32_t episode[N], prio[N];
    uint64_t seed = 7;
    for (int j = 0; j < N; ++j) {
        for (int b = 0; b < ROW; ++b) obs[j * ROW + b] = (uint8_t)splitmix(&seed);
        action[j] = j;
        reward[j] = (float)j * 0.5f;
        done[j] = (uint8_t)(j % 50 == 49);
        episode[j] = (uint32_t)(j / 50);
        step[j] = j % 50;
        prio[j] = 1u + (uint32_t)(splitmix(&seed) % 1000u);
    }
    conduit_buffer_opts o;
    conduit_buffer_opts_default(&o);
    const int64_t shape[1] = {ROW};
    conduit_buffer* buf = NULL;
    CHECK(conduit_buffer_create(CAP, shape, 1, CONDUIT_U8, &o, NULL, 0, &buf) == CONDUIT_OK, "create");

    conduit_transitions t;
    memset(&t, 0, sizeof(t));
    t.n = N;
    t.obs = dev_copy(obs, sizeof(obs));
    t.action = dev_copy(action, sizeof(action));
    t.reward = dev_copy(reward, sizeof(reward));
    t.done = dev_copy(done, sizeof(done));
    t.episode_id = dev_copy(episode, sizeof(episode));
    t.step = dev_copy(step, sizeof(step));
    t.prio = dev_copy(prio, sizeof(prio));
    CHECK(t.obs && t.action && t.reward && t.done && t.episode_id && t.step && t.prio, "device copies");
    CHECK(conduit_ingest(buf, &t, NULL) == CONDUIT_OK, "ingest");
    int64_t size = 0, head = 0;
    uint64_t total = 0;
    CHECK(conduit_buffer_stats(buf, &size, &head, &total) == CONDUIT_OK, "stats");
    CHECK(size == N && head == N && total == N, "ring state after the ingest");

    uint64_t u[BATCH];
    for (int k = 0; k < BATCH; ++k) u[k] = splitmix(&seed);
    void* u_d = dev_copy(u, sizeof(u));
    int64_t* idx_d = NULL;
    float* w_d = NULL;
    uint8_t* out_d = NULL;
    float* rew_d = NULL;
    CHECK(u_d && hipMalloc((void**)&idx_d, BATCH * 8) == hipSuccess && hipMalloc((void**)&w_d, BATCH * 4) == hipSuccess &&
              hipMalloc((void**)&out_d, BATCH * ROW) == hipSuccess && hipMalloc((void**)&rew_d, BATCH * 4) == hipSuccess,
          "output allocations");
    conduit_transform xf;
    memset(&xf, 0, sizeof(xf));
    xf.kind = CONDUIT_XF_NONE;
    conduit_learner_batch lb;
    memset(&lb, 0, sizeof(lb));
    lb.obs = out_d;
    lb.reward = rew_d;
    CHECK(conduit_sample_gather(buf, BATCH, (const uint64_t*)u_d, idx_d, w_d, &xf, &lb, NULL) == CONDUIT_OK,
          "sample_gather");
    CHECK(conduit_sync_check(buf, NULL) == CONDUIT_OK, "sync_check after sampling");
    int64_t idx[BATCH];
    float w[BATCH], rew[BATCH];
    uint8_t out[BATCH * ROW];
    CHECK(hipMemcpy(idx, idx_d, sizeof(idx), hipMemcpyDeviceToHost) == hipSuccess &&
              hipMemcpy(w, w_d, sizeof(w), hipMemcpyDeviceToHost) == hipSuccess &&
              hipMemcpy(out, out_d, sizeof(out), hipMemcpyDeviceToHost) == hipSuccess &&
              hipMemcpy(rew, rew_d, sizeof(rew), hipMemcpyDeviceToHost) == hipSuccess,
          "copies back");
    float wmax = 0.0f;
    for (int k = 0; k < BATCH; ++k) {
        CHECK(idx[k] >= 0 && idx[k] < N, "sampled index in range");
        CHECK(memcmp(out + k * ROW, obs + idx[k] * ROW, ROW) == 0, "gathered row equals the ingested bytes");
        CHECK(rew[k] == reward[idx[k]], "gathered reward");
        CHECK(w[k] > 0.0f && w[k] <= 1.0f, "importance weight in (0, 1]");
        if (w[k] > wmax) wmax = w[k];
    }
    CHECK(wmax == 1.0f, "the largest weight of the batch is 1");

    uint32_t new_prio[BATCH];
    for (int k = 0; k < BATCH; ++k) new_prio[k] = 5000u + (uint32_t)k;
    void* np_d = dev_copy(new_prio, sizeof(new_prio));
    CHECK(np_d && conduit_update_priorities(buf, idx_d, (const uint32_t*)np_d, BATCH, NULL) == CONDUIT_OK, "update");

    uint64_t img_bytes = 0;
    CHECK(conduit_buffer_checkpoint_bytes(buf, &img_bytes) == CONDUIT_OK && img_bytes > 0, "checkpoint size");
    uint8_t* img = (uint8_t*)malloc(img_bytes);
    CHECK(img && conduit_buffer_checkpoint(buf, img, img_bytes, NULL) == CONDUIT_OK, "checkpoint to host memory");
    conduit_buffer* buf2 = NULL;
    CHECK(conduit_buffer_create(CAP, shape, 1, CONDUIT_U8, &o, NULL, 0, &buf2) == CONDUIT_OK, "second buffer");
    CHECK(conduit_buffer_restore(buf2, img, img_bytes, NULL) == CONDUIT_OK, "restore");
    CHECK(conduit_buffer_stats(buf2, &size, &head, &total) == CONDUIT_OK && size == N && head == N && total == N,
          "restored ring state");
    uint32_t leaf_a[CAP], leaf_b[CAP];
    uint32_t* leaves_d = NULL;
    CHECK(hipMalloc((void**)&leaves_d, 2 * sizeof(leaf_a)) == hipSuccess, "leaf buffer");
    CHECK(conduit_buffer_read(buf, CONDUIT_COL_LEAVES, 0, 0, sizeof(leaf_a), leaves_d, NULL) == CONDUIT_OK &&
              conduit_buffer_read(buf2, CONDUIT_COL_LEAVES, 0, 0, sizeof(leaf_b), leaves_d + CAP, NULL) == CONDUIT_OK &&
              hipMemcpy(leaf_a, leaves_d, sizeof(leaf_a), hipMemcpyDeviceToHost) == hipSuccess &&
              hipMemcpy(leaf_b, leaves_d + CAP, sizeof(leaf_b), hipMemcpyDeviceToHost) == hipSuccess,
          "leaf reads");
    CHECK(memcmp(leaf_a, leaf_b, sizeof(leaf_a)) == 0, "restored leaves");
    free(img);
    conduit_buffer_destroy(buf2);
    conduit_buffer_destroy(buf);
    printf("c consumer ok\n");
    return 0;
}
