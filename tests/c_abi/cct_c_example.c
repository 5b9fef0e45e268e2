/* A plain C client of the library's C ABI (include/cct.h): no Python, no torch.  It
 * builds the hand-worked tree W1 (tests/golden/W1.txt) from device buffers, merges one
 * more batch, looks up two paths and prints every result as text, which the GPU test
 * compares with the oracle.  Exit status 0 on success, 1 with a message on any failure. */
#include <hip/hip_runtime_api.h>
#include <inttypes.h>
#include <stdio.h>
#include <stdlib.h>

#include "cct.h"

#define CHECK_HIP(x)                                                        \
  do {                                                                      \
    if ((x) != hipSuccess) {                                                \
      fprintf(stderr, "HIP error at line %d\n", __LINE__);                  \
      return 1;                                                             \
    }                                                                       \
  } while (0)
#define CHECK_CCT(x)                                                        \
  do {                                                                      \
    if ((x) != CCT_OK) {                                                    \
      fprintf(stderr, "cct error at line %d: %s\n", __LINE__, cct_last_error()); \
      return 1;                                                             \
    }                                                                       \
  } while (0)

/* Allocates `bytes` of device memory and, when `host` is given, copies it there. */
static int to_device(const void *host, size_t bytes, void **dev) {
  hipError_t e = hipMalloc(dev, bytes ? bytes : 8);
  if (e != hipSuccess) {
    fprintf(stderr, "hipMalloc(%zu): %s\n", bytes, hipGetErrorString(e));
    return 1;
  }
  if (host && bytes && (e = hipMemcpy(*dev, host, bytes, hipMemcpyHostToDevice)) != hipSuccess) {
    fprintf(stderr, "hipMemcpy(%zu): %s\n", bytes, hipGetErrorString(e));
    return 1;
  }
  return 0;
}

static int print_tree(const char *tag, const cct_tree *t) {
  int64_t u = 0, d = 0;
  int32_t m = 0;
  CHECK_CCT(cct_info(t, &u, &m, &d));
  uint32_t *parent = malloc(u * 4), *frame = malloc(u * 4), *depth = malloc(u * 4);
  uint64_t *excl = malloc(u * m * 8), *incl = malloc(u * m * 8);
  if (!parent || !frame || !depth || !excl || !incl) return 1;
  CHECK_CCT(cct_export(t, NULL, parent, frame, depth, excl, incl));  /* host destinations */
  printf("%s %" PRId64 " %" PRId64 "\n", tag, u, d);
  for (int64_t v = 0; v < u; ++v)
    printf("N %u %u %u %" PRIu64 " %" PRIu64 "\n", parent[v], frame[v], depth[v], excl[v * m], incl[v * m]);
  free(parent); free(frame); free(depth); free(excl); free(incl);
  return 0;
}

int main(void) {
  /* W1: events [1,2]:5 [1,2,3]:3 [1]:2 [4]:7 [1,3]:1 */
  const int64_t off[] = {0, 2, 5, 6, 7, 9};
  const uint32_t fr[] = {1, 2, 1, 2, 3, 1, 4, 1, 3};
  const uint64_t w[] = {5, 3, 2, 7, 1};
  /* a second batch: [1,2]:4 and [4,5]:6 */
  const int64_t off2[] = {0, 2, 4};
  const uint32_t fr2[] = {1, 2, 4, 5};
  const uint64_t w2[] = {4, 6};
  /* queries: [1,2] (a node) and [2] (absent) */
  const int64_t qoff[] = {0, 2, 3};
  const uint32_t qfr[] = {1, 2, 2};
  void *d_off, *d_fr, *d_w, *d_off2, *d_fr2, *d_w2, *d_qoff, *d_qfr, *d_ids, *d_incl;
  if (to_device(off, sizeof off, &d_off) || to_device(fr, sizeof fr, &d_fr) || to_device(w, sizeof w, &d_w) ||
      to_device(off2, sizeof off2, &d_off2) || to_device(fr2, sizeof fr2, &d_fr2) ||
      to_device(w2, sizeof w2, &d_w2) || to_device(qoff, sizeof qoff, &d_qoff) ||
      to_device(qfr, sizeof qfr, &d_qfr) || to_device(NULL, 16, &d_ids) || to_device(NULL, 16, &d_incl)) {
    fprintf(stderr, "device allocation or copy failed\n");
    return 1;
  }
  cct_paths batch = {5, 9, 1, (const int64_t *)d_off, (const uint32_t *)d_fr, (const uint64_t *)d_w};
  cct_tree *tree = NULL;
  CHECK_CCT(cct_build(&batch, NULL, &tree));
  if (print_tree("BUILD", tree)) return 1;
  cct_paths batch2 = {2, 4, 1, (const int64_t *)d_off2, (const uint32_t *)d_fr2, (const uint64_t *)d_w2};
  CHECK_CCT(cct_merge(tree, &batch2, NULL));
  if (print_tree("MERGE", tree)) return 1;
  cct_paths queries = {2, 3, 1, (const int64_t *)d_qoff, (const uint32_t *)d_qfr, NULL};
  CHECK_CCT(cct_query(tree, &queries, NULL, (int64_t *)d_ids, NULL, (uint64_t *)d_incl));
  int64_t ids[2];
  uint64_t incl[2];
  CHECK_HIP(hipMemcpy(ids, d_ids, sizeof ids, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(incl, d_incl, sizeof incl, hipMemcpyDeviceToHost));
  printf("Q %" PRId64 " %" PRIu64 " %" PRId64 " %" PRIu64 "\n", ids[0], incl[0], ids[1], incl[1]);
  cct_free(tree);
  hipFree(d_off); hipFree(d_fr); hipFree(d_w); hipFree(d_off2); hipFree(d_fr2); hipFree(d_w2);
  hipFree(d_qoff); hipFree(d_qfr); hipFree(d_ids); hipFree(d_incl);
  return 0;
}
