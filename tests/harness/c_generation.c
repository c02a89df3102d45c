/* One ES generation driven from C through the library's public header and
 * the HIP runtime alone (no Python in the loop): G = 4 members over two bf16
 * tensors, the second 2-byte aligned only -- apply the first member, then
 * swap each member for the next, then revert the last member inside the
 * update (Section 3; Appendix D.6 order), and checksum the result.
 *
 *   c_generation IN PERTURBED FINAL N0 N1 [MASTERS]
 *
 * IN holds N0 + N1 bf16 bit patterns (tensor 0, then tensor 1, little
 * endian); PERTURBED receives both tensors after the first member is
 * applied, FINAL after the update.  With MASTERS the generation runs over
 * binary32 masters instead, initialised to IN's values: each member is
 * applied from them (es_perturb_master, no revert), the update goes into
 * them (ES_UPDATE_MASTER), and MASTERS receives their N0 + N1 binary32 bit
 * patterns.  Prints the radius, the z-scores, the status word and the plan
 * checksum on stdout.  Exits non-zero, naming the failing call, on any
 * error. */
#include <hip/hip_runtime_api.h>
#include <inttypes.h>
#include <stdio.h>
#include <stdlib.h>

#include "esopt.h"

#define G 4

static int check_es(int rc, const char* what) {
    if (rc != ES_OK) {
        fprintf(stderr, "%s: %s: %s\n", what, es_strerror(rc), es_last_error());
        return 1;
    }
    return 0;
}

static int check_hip(hipError_t e, const char* what) {
    if (e != hipSuccess) {
        fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
        return 1;
    }
    return 0;
}

/* Both tensors, device to the file at path. */
static int save(const char* path, const uint16_t* d0, uint64_t n0, const uint16_t* d1,
                uint64_t n1, uint16_t* host) {
    if (check_hip(hipMemcpy(host, d0, 2 * n0, hipMemcpyDeviceToHost), "hipMemcpy") ||
        check_hip(hipMemcpy(host + n0, d1, 2 * n1, hipMemcpyDeviceToHost), "hipMemcpy"))
        return 1;
    FILE* f = fopen(path, "wb");
    if (f == NULL || fwrite(host, 2, n0 + n1, f) != n0 + n1) {
        fprintf(stderr, "cannot write %s\n", path);
        if (f) fclose(f);
        return 1;
    }
    return fclose(f) != 0;
}

int main(int argc, char** argv) {
    if (argc != 6 && argc != 7) {
        fprintf(stderr, "usage: %s IN PERTURBED FINAL N0 N1 [MASTERS]\n", argv[0]);
        return 2;
    }
    const int with_masters = argc == 7;
    const uint64_t n0 = strtoull(argv[4], NULL, 10), n1 = strtoull(argv[5], NULL, 10);
    const uint64_t n = n0 + n1;
    uint16_t* host = malloc(2 * n);
    FILE* f = fopen(argv[1], "rb");
    if (host == NULL || f == NULL || fread(host, 2, n, f) != n) {
        fprintf(stderr, "cannot read %s\n", argv[1]);
        return 1;
    }
    fclose(f);

    /* tensor 0 at the allocation's start; tensor 1 one element past its
     * end, so only 2-byte aligned */
    uint16_t* buf = NULL;
    if (check_hip(hipMalloc((void**)&buf, 2 * (n + 1)), "hipMalloc")) return 1;
    uint16_t* d0 = buf;
    uint16_t* d1 = buf + n0 + 1;
    if (check_hip(hipMemcpy(d0, host, 2 * n0, hipMemcpyHostToDevice), "hipMemcpy") ||
        check_hip(hipMemcpy(d1, host + n0, 2 * n1, hipMemcpyHostToDevice), "hipMemcpy"))
        return 1;

    es_tensor_t tensors[2] = {{d0, n0, 0u, 0u}, {d1, n1, 5u, 0u}};
    es_plan_t* plan = NULL;
    if (check_es(es_plan_create(tensors, 2, &plan), "es_plan_create")) return 1;

    const uint64_t seeds[G] = {100, 101, 102, 103};
    const int32_t signs[G] = {1, 1, 1, 1};
    const float rewards[G] = {0.3f, 0.9f, 0.1f, 0.6f};   /* stand-ins for the evaluations */
    const float sigma = (float)es_sigma_cosine(1e-3, 1e-4, 3, 100);
    hipStream_t s = NULL;
    if (check_hip(hipStreamCreate(&s), "hipStreamCreate")) return 1;

    /* binary32 masters of both tensors, one allocation each, set to IN's
     * values (a bf16 pattern shifted up 16 bits is that value in binary32) */
    float* m0 = NULL;
    float* m1 = NULL;
    uint32_t* mhost = NULL;
    if (with_masters) {
        mhost = malloc(4 * n);
        if (mhost == NULL) return 1;
        for (uint64_t j = 0; j < n; ++j) mhost[j] = (uint32_t)host[j] << 16;
        void* masters[2];
        if (check_hip(hipMalloc((void**)&m0, 4 * n0), "hipMalloc") ||
            check_hip(hipMalloc((void**)&m1, 4 * n1), "hipMalloc") ||
            check_hip(hipMemcpy(m0, mhost, 4 * n0, hipMemcpyHostToDevice), "hipMemcpy") ||
            check_hip(hipMemcpy(m1, mhost + n0, 4 * n1, hipMemcpyHostToDevice), "hipMemcpy"))
            return 1;
        masters[0] = m0;
        masters[1] = m1;
        if (check_es(es_plan_set_master(plan, masters, 2), "es_plan_set_master")) return 1;
    }

    if (with_masters) {
        if (check_es(es_perturb_master(plan, seeds[0], signs[0], sigma, s), "es_perturb_master"))
            return 1;
    } else if (check_es(es_perturb(plan, seeds[0], signs[0], sigma, s), "es_perturb")) {
        return 1;
    }
    if (check_hip(hipStreamSynchronize(s), "hipStreamSynchronize") ||
        save(argv[2], d0, n0, d1, n1, host))
        return 1;
    for (int i = 1; i < G; ++i) {
        const int rc = with_masters
                           ? es_perturb_master(plan, seeds[i], signs[i], sigma, s)
                           : es_swap(plan, seeds[i - 1], signs[i - 1], sigma, seeds[i], signs[i],
                                     sigma, s);
        if (check_es(rc, with_masters ? "es_perturb_master" : "es_swap")) return 1;
    }

    float* d_rewards = NULL;
    float* d_z = NULL;
    int32_t* d_status = NULL;
    uint64_t* d_sum = NULL;
    if (check_hip(hipMalloc((void**)&d_rewards, sizeof rewards), "hipMalloc") ||
        check_hip(hipMalloc((void**)&d_z, sizeof rewards), "hipMalloc") ||
        check_hip(hipMalloc((void**)&d_status, sizeof(int32_t)), "hipMalloc") ||
        check_hip(hipMalloc((void**)&d_sum, sizeof(uint64_t)), "hipMalloc") ||
        check_hip(hipMemcpy(d_rewards, rewards, sizeof rewards, hipMemcpyHostToDevice),
                  "hipMemcpy"))
        return 1;
    es_update_opts_t opts = {5e-4f, sigma, 1e-8f, with_masters ? ES_UPDATE_MASTER : 0u, 0u};
    /* with masters the update rewrites every bf16 value: no revert first */
    const int rc = with_masters
                       ? es_update(plan, seeds, signs, d_rewards, G, &opts, d_z, d_status, s)
                       : es_restore_update(plan, seeds[G - 1], signs[G - 1], sigma, seeds, signs,
                                           d_rewards, G, &opts, d_z, d_status, s);
    if (check_es(rc, with_masters ? "es_update" : "es_restore_update") ||
        check_es(es_plan_checksum(plan, d_sum, s), "es_plan_checksum") ||
        check_hip(hipStreamSynchronize(s), "hipStreamSynchronize") ||
        save(argv[3], d0, n0, d1, n1, host))
        return 1;

    float z[G];
    int32_t status = -1;
    uint64_t sum = 0;
    if (check_hip(hipMemcpy(z, d_z, sizeof z, hipMemcpyDeviceToHost), "hipMemcpy") ||
        check_hip(hipMemcpy(&status, d_status, sizeof status, hipMemcpyDeviceToHost),
                  "hipMemcpy") ||
        check_hip(hipMemcpy(&sum, d_sum, sizeof sum, hipMemcpyDeviceToHost), "hipMemcpy"))
        return 1;
    printf("sigma %.9g\n", (double)sigma);
    printf("z %.9g %.9g %.9g %.9g\n", (double)z[0], (double)z[1], (double)z[2], (double)z[3]);
    printf("status %d\n", (int)status);
    printf("checksum %" PRIu64 "\n", sum);

    if (with_masters) {
        FILE* mf = NULL;
        if (check_hip(hipMemcpy(mhost, m0, 4 * n0, hipMemcpyDeviceToHost), "hipMemcpy") ||
            check_hip(hipMemcpy(mhost + n0, m1, 4 * n1, hipMemcpyDeviceToHost), "hipMemcpy"))
            return 1;
        mf = fopen(argv[6], "wb");
        if (mf == NULL || fwrite(mhost, 4, n, mf) != n || fclose(mf) != 0) {
            fprintf(stderr, "cannot write %s\n", argv[6]);
            return 1;
        }
    }

    if (check_es(es_plan_destroy(plan), "es_plan_destroy")) return 1;
    hipFree(m0);
    hipFree(m1);
    free(mhost);
    hipFree(d_rewards);
    hipFree(d_z);
    hipFree(d_status);
    hipFree(d_sum);
    hipFree(buf);
    hipStreamDestroy(s);
    free(host);
    return 0;
}
