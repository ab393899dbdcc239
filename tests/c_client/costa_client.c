/* A plain C99 client of the library, compiled against include/costa.h with a
 * C compiler and linked against libcosta_mi355x.so and the HIP runtime: the
 * tests use it to check that the header, the library and the Python binding
 * agree (struct layouts, enum values, results), independently of ctypes.
 *
 *   costa_client host <A: M N mb nb prow pcol ro bo> <B: same> <op>
 *       host-only entry points; prints one line per result
 *   costa_client gpu <dir> <A> <B> <op> <alpha> <beta>
 *       fp64 transform A <- alpha*op(B) + beta*A on the first device:
 *       reads dir/b.bin and dir/a.bin (the local buffers of ranks 0..P-1,
 *       one after another), writes dir/out.bin (A after the transform)
 *
 * Built with -DCOSTA_CLIENT_NO_MAIN -shared, the same code is a library whose
 * costa_client_host() and costa_client_gpu() do what "host" and "gpu" do, for
 * callers that must stay in one process (a process that has already used the
 * GPU does not start others).
 *
 * ro / bo: 'r' (row-major) or 'c' (column-major) rank order and block
 * storage order of a block-cyclic layout.  Exit status 0 on success. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "costa.h"

static int fail_status(const char* what, costa_status st) {
  fprintf(stderr, "%s: %s (%s)\n", what, costa_status_string(st), costa_last_error());
  return 1;
}

#define CHECK(call)                                  \
  do {                                               \
    costa_status st_ = (call);                       \
    if (st_ != COSTA_SUCCESS) return fail_status(#call, st_); \
  } while (0)

#define HIP_CHECK(call)                                                   \
  do {                                                                    \
    hipError_t e_ = (call);                                               \
    if (e_ != hipSuccess) {                                               \
      fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));          \
      return 1;                                                           \
    }                                                                     \
  } while (0)

static costa_order order_of(const char* s) { return s[0] == 'r' ? COSTA_ROW_MAJOR : COSTA_COL_MAJOR; }

static costa_op op_of(const char* s) {
  if (s[0] == 'T') return COSTA_OP_T;
  if (s[0] == 'C') return COSTA_OP_C;
  return COSTA_OP_N;
}

/* 8 arguments: M N mb nb prow pcol rank_order block_order */
static costa_status make_layout(char** a, costa_layout* out) {
  return costa_layout_create_block_cyclic(atoll(a[0]), atoll(a[1]), atoll(a[2]), atoll(a[3]), atoi(a[4]),
                                          atoi(a[5]), order_of(a[6]), order_of(a[7]), out);
}

int costa_client_host(char** a, char** b, const char* ops);

int costa_client_host(char** a, char** b, const char* ops) {
  costa_layout A = NULL, B = NULL;
  CHECK(make_layout(a, &A));
  CHECK(make_layout(b, &B));
  const int32_t P = atoi(a[4]) * atoi(a[5]);
  for (int32_t r = 0; r < P; ++r) {
    int64_t na = 0, nb = 0;
    CHECK(costa_layout_local_elems(A, r, &na));
    CHECK(costa_layout_local_elems(B, r, &nb));
    printf("local %d %lld %lld\n", r, (long long)na, (long long)nb);
  }
  costa_transform_desc d;
  memset(&d, 0, sizeof d);
  d.op = op_of(ops);
  d.A = A;
  d.B = B;
  costa_stats s;
  CHECK(costa_plan_stats(COSTA_R64, 1, &d, NULL, &s));
  printf("stats %lld %lld %lld %lld %lld %lld %lld %lld %lld %lld %d %d %d %d\n", (long long)s.total_elems,
         (long long)s.local_elems, (long long)s.remote_elems, (long long)s.model_bytes, (long long)s.message_bytes,
         (long long)s.workspace_bytes, (long long)s.overlay_blocks, (long long)s.pack_bytes,
         (long long)s.unpack_bytes, (long long)s.direct_bytes, s.waves, s.pieces_pack, s.pieces_unpack,
         s.pieces_direct);
  int64_t count = 0;
  CHECK(costa_plan_export(COSTA_R64, 1, &d, NULL, NULL, 0, &count));
  costa_piece_info* pieces = (costa_piece_info*)calloc((size_t)(count > 0 ? count : 1), sizeof *pieces);
  if (!pieces) return 1;
  CHECK(costa_plan_export(COSTA_R64, 1, &d, NULL, pieces, count, &count));
  /* every field of every rectangle, folded into one checksum the test recomputes */
  uint64_t h = 1469598103934665603ull;
  for (int64_t k = 0; k < count; ++k) {
    const costa_piece_info* p = &pieces[k];
    const int64_t f[] = {p->kind,   p->wave,    p->group,   p->src_off, p->dst_off, p->src_ld,
                         p->dst_ld, p->src_buf, p->dst_buf, p->nx,      p->ny,      p->item,
                         p->flags,  p->ntasks,  p->tile_x,  p->tile_y,  p->launch,  p->wide_group,
                         p->wide_ntasks};
    for (size_t i = 0; i < sizeof f / sizeof f[0]; ++i) h = (h ^ (uint64_t)f[i]) * 1099511628211ull;
  }
  printf("pieces %lld %llu\n", (long long)count, (unsigned long long)h);
  free(pieces);

  /* relabeling of a fixed 3 x 3 volume matrix, exact and greedy */
  const int64_t V[9] = {0, 0, 0, 5, 0, 4, 4, 0, 0};
  int32_t sigma[3];
  int64_t kept_id = 0, kept = 0;
  CHECK(costa_relabel(3, V, sigma, &kept_id, &kept));
  printf("relabel %d %d %d %lld %lld\n", sigma[0], sigma[1], sigma[2], (long long)kept_id, (long long)kept);
  double before = 0, after = 0;
  CHECK(costa_relabel_cost(3, V, 1.0, NULL, NULL, COSTA_RELABEL_GREEDY, sigma, &before, &after));
  printf("greedy %d %d %d %.1f %.1f\n", sigma[0], sigma[1], sigma[2], before, after);

  /* an invalid argument: status code and a message */
  costa_layout bad = NULL;
  costa_status st = costa_layout_create_block_cyclic(10, 10, 0, 2, 1, 1, COSTA_ROW_MAJOR, COSTA_COL_MAJOR, &bad);
  printf("error %d %d\n", (int)st, (int)(strlen(costa_last_error()) > 0));
  st = costa_transform(COSTA_R64, (costa_op)7, NULL, NULL, A, NULL, B, NULL, NULL, NULL);
  printf("error %d\n", (int)st);

  CHECK(costa_layout_destroy(A));
  CHECK(costa_layout_destroy(B));
  return 0;
}

static int read_all(const char* path, double* dst, size_t n) {
  FILE* f = fopen(path, "rb");
  if (!f) return 1;
  size_t got = n ? fread(dst, sizeof(double), n, f) : 0;
  fclose(f);
  return got == n ? 0 : 1;
}

int costa_client_gpu(const char* dir, char** a, char** b, const char* ops, double alpha, double beta);

int costa_client_gpu(const char* dir, char** a, char** b, const char* ops, double alpha, double beta) {
  costa_layout A = NULL, B = NULL;
  CHECK(make_layout(a, &A));
  CHECK(make_layout(b, &B));
  const int32_t P = atoi(a[4]) * atoi(a[5]);
  if (P <= 0 || P > 4096 || atoi(b[4]) * atoi(b[5]) != P) return 1;
  int64_t* na = (int64_t*)calloc((size_t)P, sizeof(int64_t));
  int64_t* nb = (int64_t*)calloc((size_t)P, sizeof(int64_t));
  void** dA = (void**)calloc((size_t)P, sizeof(void*));
  const void** dB = (const void**)calloc((size_t)P, sizeof(void*));
  if (!na || !nb || !dA || !dB) return 1;
  int64_t ta = 0, tb = 0;
  for (int32_t r = 0; r < P; ++r) {
    CHECK(costa_layout_local_elems(A, r, &na[r]));
    CHECK(costa_layout_local_elems(B, r, &nb[r]));
    ta += na[r];
    tb += nb[r];
  }
  double* ha = (double*)malloc((size_t)(ta > 0 ? ta : 1) * sizeof(double));
  double* hb = (double*)malloc((size_t)(tb > 0 ? tb : 1) * sizeof(double));
  if (!ha || !hb) return 1;
  char path[4096];
  snprintf(path, sizeof path, "%s/a.bin", dir);
  if (read_all(path, ha, (size_t)ta)) return 1;
  snprintf(path, sizeof path, "%s/b.bin", dir);
  if (read_all(path, hb, (size_t)tb)) return 1;
  int64_t oa = 0, ob = 0;
  for (int32_t r = 0; r < P; ++r) {
    void* p = NULL;
    if (na[r]) {
      HIP_CHECK(hipMalloc(&p, (size_t)na[r] * sizeof(double)));
      HIP_CHECK(hipMemcpy(p, ha + oa, (size_t)na[r] * sizeof(double), hipMemcpyHostToDevice));
    }
    dA[r] = p;
    oa += na[r];
    p = NULL;
    if (nb[r]) {
      HIP_CHECK(hipMalloc(&p, (size_t)nb[r] * sizeof(double)));
      HIP_CHECK(hipMemcpy(p, hb + ob, (size_t)nb[r] * sizeof(double), hipMemcpyHostToDevice));
    }
    dB[r] = p;
    ob += nb[r];
  }
  hipStream_t stream;
  HIP_CHECK(hipStreamCreate(&stream));
  CHECK(costa_transform(COSTA_R64, op_of(ops), &alpha, &beta, A, dA, B, dB, NULL, stream));
  HIP_CHECK(hipStreamSynchronize(stream));
  oa = 0;
  for (int32_t r = 0; r < P; ++r) {
    if (na[r]) HIP_CHECK(hipMemcpy(ha + oa, dA[r], (size_t)na[r] * sizeof(double), hipMemcpyDeviceToHost));
    oa += na[r];
  }
  snprintf(path, sizeof path, "%s/out.bin", dir);
  FILE* f = fopen(path, "wb");
  if (!f || (ta && fwrite(ha, sizeof(double), (size_t)ta, f) != (size_t)ta)) return 1;
  fclose(f);
  for (int32_t r = 0; r < P; ++r) {
    if (dA[r]) HIP_CHECK(hipFree(dA[r]));
    if (dB[r]) HIP_CHECK(hipFree((void*)dB[r]));
  }
  HIP_CHECK(hipStreamDestroy(stream));
  CHECK(costa_layout_destroy(A));
  CHECK(costa_layout_destroy(B));
  free(na);
  free(nb);
  free(dA);
  free(dB);
  free(ha);
  free(hb);
  return 0;
}

#ifndef COSTA_CLIENT_NO_MAIN
int main(int argc, char** argv) {
  if (argc == 19 && strcmp(argv[1], "host") == 0) return costa_client_host(argv + 2, argv + 10, argv[18]);
  if (argc == 22 && strcmp(argv[1], "gpu") == 0) {
    const int rc = costa_client_gpu(argv[2], argv + 3, argv + 11, argv[19], atof(argv[20]), atof(argv[21]));
    if (rc != 0) return rc;
    CHECK(costa_finalize()); /* a program that is done with the library releases its caches */
    printf("ok\n");
    return 0;
  }
  fprintf(stderr, "usage: costa_client host <A x8> <B x8> <op> | gpu <dir> <A x8> <B x8> <op> <alpha> <beta>\n");
  return 2;
}
#endif
