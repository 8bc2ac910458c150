/*
 * A plain C client of the library: the C ABI of include/pda.h as an engine
 * written in C would use it, with device memory and streams from the HIP
 * runtime's C API and no Python or torch anywhere.
 *
 *   pda_client errors     argument checks that return before any HIP call
 *                         (runs without a GPU), for the pointer and the
 *                         tensor-descriptor entry points; prints "ok <check>"
 *                         lines
 *   pda_client run DIR    decode attention on the device: reads DIR/meta.txt
 *                         ("batch hq hkv head_dim page_size num_pages maxp
 *                         scale") and the raw little-endian arrays DIR/q.bin,
 *                         k.bin, v.bin (bf16 bits), bt.bin and lens.bin
 *                         (int32); runs the call on a created stream after
 *                         reserving its workspace, and again on the null
 *                         stream, checks that both outputs are bitwise
 *                         equal, and writes the first to DIR/out.bin; then
 *                         captures the call on the created stream into a
 *                         HIP graph and checks that three replays (output
 *                         cleared in between) reproduce it bitwise
 *
 * Exit status 0 when every check holds.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "pda.h"

static int failures = 0;

static void expect(const char* what, int got, int want) {
  if (got == want) {
    printf("ok %s\n", what);
  } else {
    printf("FAIL %s: status %d, expected %d (%s)\n", what, got, want, pda_last_error());
    ++failures;
  }
}

/* A dense row-major descriptor of `ndim` extents. */
static pda_tensor desc(void* data, int32_t dtype, int32_t ndim, const int64_t* shape) {
  pda_tensor t;
  memset(&t, 0, sizeof t);
  t.data = data;
  t.dtype = dtype;
  t.ndim = ndim;
  int64_t acc = 1;
  for (int i = ndim - 1; i >= 0; --i) {
    t.shape[i] = shape[i];
    t.stride[i] = acc;
    acc *= shape[i];
  }
  return t;
}

/* The descriptor entry point with one argument spoiled at a time: each
   validation error is returned before any HIP call. */
static void run_descriptor_errors(void* p) {
  const int64_t qs[3] = {2, 32, 128}, ks[4] = {64, 16, 8, 128}, bs[2] = {2, 8}, ls[1] = {2};
  const pda_tensor q = desc(p, PDA_DTYPE_BF16, 3, qs), k = desc(p, PDA_DTYPE_BF16, 4, ks);
  const pda_tensor bt = desc(p, PDA_DTYPE_I32, 2, bs), lens = desc(p, PDA_DTYPE_I32, 1, ls);
  pda_tensor t;

  expect("desc null descriptor", paged_decode_attention_desc(NULL, &k, &k, &bt, &lens, &q, 0.088f, NULL),
         PDA_ERR_NULL);
  t = desc(NULL, PDA_DTYPE_BF16, 4, ks);
  expect("desc null data", paged_decode_attention_desc(&q, &t, &k, &bt, &lens, &q, 0.088f, NULL), PDA_ERR_NULL);
  t = desc(p, PDA_DTYPE_F16, 3, qs);
  expect("desc fp16 q", paged_decode_attention_desc(&t, &k, &k, &bt, &lens, &q, 0.088f, NULL), PDA_ERR_DTYPE);
  t = desc(p, PDA_DTYPE_I64, 1, ls);
  expect("desc int64 lengths", paged_decode_attention_desc(&q, &k, &k, &bt, &t, &q, 0.088f, NULL), PDA_ERR_DTYPE);
  t = desc(p, PDA_DTYPE_BF16, 2, qs);
  expect("desc q rank", paged_decode_attention_desc(&t, &k, &k, &bt, &lens, &q, 0.088f, NULL), PDA_ERR_SHAPE);
  {
    const int64_t bs3[2] = {3, 8};
    t = desc(p, PDA_DTYPE_I32, 2, bs3);
    expect("desc block_table rows", paged_decode_attention_desc(&q, &k, &k, &t, &lens, &q, 0.088f, NULL),
           PDA_ERR_SHAPE);
  }
  {
    const int64_t q30[3] = {2, 30, 128};
    t = desc(p, PDA_DTYPE_BF16, 3, q30);
    expect("desc heads not a multiple", paged_decode_attention_desc(&t, &k, &k, &bt, &lens, &t, 0.088f, NULL),
           PDA_ERR_SHAPE);
  }
  {
    const int64_t q96[3] = {2, 32, 96}, k96[4] = {64, 16, 8, 96};
    const pda_tensor a = desc(p, PDA_DTYPE_BF16, 3, q96), c = desc(p, PDA_DTYPE_BF16, 4, k96);
    expect("desc head_dim 96", paged_decode_attention_desc(&a, &c, &c, &bt, &lens, &a, 0.088f, NULL),
           PDA_ERR_UNSUPPORTED);
  }
  {
    const int64_t k24[4] = {64, 24, 8, 128};
    t = desc(p, PDA_DTYPE_BF16, 4, k24);
    expect("desc page_size 24", paged_decode_attention_desc(&q, &t, &t, &bt, &lens, &q, 0.088f, NULL),
           PDA_ERR_UNSUPPORTED);
  }
  t = q;  /* a transposed view: heads and features swapped in memory */
  t.stride[1] = 1;
  t.stride[2] = 32;
  expect("desc transposed q", paged_decode_attention_desc(&t, &k, &k, &bt, &lens, &q, 0.088f, NULL),
         PDA_ERR_LAYOUT);
  t = bt;  /* rows of a wider table */
  t.stride[0] = 16;
  expect("desc padded block_table", paged_decode_attention_desc(&q, &k, &k, &t, &lens, &q, 0.088f, NULL),
         PDA_ERR_LAYOUT);
  expect("desc nan scale", paged_decode_attention_desc(&q, &k, &k, &bt, &lens, &q, nanf(""), NULL),
         PDA_ERR_SCALE);
}

static int run_errors(void) {
  /* Any 16-byte aligned non-NULL address: these calls must reject their
     arguments before touching memory or the device. */
  void* p = (void*)(uintptr_t)0x1000;
  const int32_t* ip = (const int32_t*)p;
  expect("null q", paged_decode_attention(NULL, p, p, ip, ip, p, 2, 32, 8, 128, 16, 64, 8, 0.088f, NULL),
         PDA_ERR_NULL);
  if (failures == 0 && strlen(pda_last_error()) == 0) {
    printf("FAIL empty error message\n");
    ++failures;
  }
  expect("head_dim 96", paged_decode_attention(p, p, p, ip, ip, p, 2, 32, 8, 96, 16, 64, 8, 0.088f, NULL),
         PDA_ERR_UNSUPPORTED);
  expect("group 32", paged_decode_attention(p, p, p, ip, ip, p, 2, 64, 2, 128, 16, 64, 8, 0.088f, NULL),
         PDA_ERR_UNSUPPORTED);
  expect("heads not a multiple", paged_decode_attention(p, p, p, ip, ip, p, 2, 30, 8, 128, 16, 64, 8, 0.088f, NULL),
         PDA_ERR_SHAPE);
  expect("misaligned q",
         paged_decode_attention((void*)(uintptr_t)0x1008, p, p, ip, ip, p, 2, 32, 8, 128, 16, 64, 8, 0.088f, NULL),
         PDA_ERR_ALIGN);
  expect("nan scale", paged_decode_attention(p, p, p, ip, ip, p, 2, 32, 8, 128, 16, 64, 8, nanf(""), NULL),
         PDA_ERR_SCALE);
  expect("empty batch", paged_decode_attention(NULL, NULL, NULL, NULL, NULL, NULL, 0, 32, 8, 128, 16, 64, 8, 0.088f,
                                               NULL),
         PDA_OK);
  if (strlen(pda_last_error()) != 0) {
    printf("FAIL error message not cleared by a successful call\n");
    ++failures;
  }
  expect("version", pda_version(), PDA_VERSION);
  run_descriptor_errors(p);

  int32_t grid = 0, waves = 0;
  int64_t ws = 0;
  expect("plan", pda_plan(4, 64, 8, 128, 16, 8192, 256, &grid, &waves, &ws), PDA_OK);
  if (grid != 256 || waves != 256 * 8 || ws <= 0) {
    printf("FAIL plan: grid %d waves %d workspace %lld\n", grid, waves, (long long)ws);
    ++failures;
  } else {
    printf("ok plan shape: grid %d waves %d workspace %lld\n", grid, waves, (long long)ws);
  }
  return failures ? 1 : 0;
}

#define HIP_OK(call)                                                              \
  do {                                                                            \
    hipError_t e_ = (call);                                                       \
    if (e_ != hipSuccess) {                                                       \
      fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));          \
      exit(2);                                                                    \
    }                                                                             \
  } while (0)

/* Reads DIR/name into a new host buffer of exactly `bytes` bytes. */
static void* read_file(const char* dir, const char* name, size_t bytes) {
  char path[4096];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE* f = fopen(path, "rb");
  if (!f) {
    fprintf(stderr, "cannot open %s\n", path);
    exit(2);
  }
  void* buf = malloc(bytes ? bytes : 1);
  if (!buf || fread(buf, 1, bytes, f) != bytes || fgetc(f) != EOF) {
    fprintf(stderr, "%s does not hold %zu bytes\n", path, bytes);
    exit(2);
  }
  fclose(f);
  return buf;
}

static void* to_device(const void* host, size_t bytes) {
  void* dev = NULL;
  HIP_OK(hipMalloc(&dev, bytes ? bytes : 16));
  if (bytes) HIP_OK(hipMemcpy(dev, host, bytes, hipMemcpyHostToDevice));
  return dev;
}

static int run_device(const char* dir) {
  char path[4096];
  snprintf(path, sizeof path, "%s/meta.txt", dir);
  FILE* f = fopen(path, "r");
  if (!f) {
    fprintf(stderr, "cannot open %s\n", path);
    return 2;
  }
  int batch, hq, hkv, d, page, num_pages, maxp;
  float scale;
  if (fscanf(f, "%d %d %d %d %d %d %d %f", &batch, &hq, &hkv, &d, &page, &num_pages, &maxp, &scale) != 8) {
    fprintf(stderr, "bad meta.txt\n");
    return 2;
  }
  fclose(f);
  const size_t q_bytes = (size_t)batch * hq * d * 2;
  const size_t kv_bytes = (size_t)num_pages * page * hkv * d * 2;
  const size_t bt_bytes = (size_t)batch * maxp * 4;
  const size_t lens_bytes = (size_t)batch * 4;

  void* hq_ = read_file(dir, "q.bin", q_bytes);
  void* hk = read_file(dir, "k.bin", kv_bytes);
  void* hv = read_file(dir, "v.bin", kv_bytes);
  void* hbt = read_file(dir, "bt.bin", bt_bytes);
  void* hlens = read_file(dir, "lens.bin", lens_bytes);
  void* q = to_device(hq_, q_bytes);
  void* k = to_device(hk, kv_bytes);
  void* v = to_device(hv, kv_bytes);
  int32_t* bt = (int32_t*)to_device(hbt, bt_bytes);
  int32_t* lens = (int32_t*)to_device(hlens, lens_bytes);
  void* out1 = NULL;
  void* out2 = NULL;
  HIP_OK(hipMalloc(&out1, q_bytes));
  HIP_OK(hipMalloc(&out2, q_bytes));
  HIP_OK(hipMemset(out1, 0xFF, q_bytes)); /* NaN bf16 bits: every row must be written */
  HIP_OK(hipMemset(out2, 0xFF, q_bytes));

  hipStream_t st;
  HIP_OK(hipStreamCreate(&st));
  expect("workspace reserve", pda_workspace_reserve(batch, hq, hkv, d, page, maxp, st), PDA_OK);
  expect("attention on a stream",
         paged_decode_attention(q, k, v, bt, lens, out1, batch, hq, hkv, d, page, num_pages, maxp, scale, st),
         PDA_OK);
  expect("attention on the null stream",
         paged_decode_attention(q, k, v, bt, lens, out2, batch, hq, hkv, d, page, num_pages, maxp, scale, NULL),
         PDA_OK);
  HIP_OK(hipStreamSynchronize(st));
  HIP_OK(hipDeviceSynchronize());

  unsigned char* o1 = (unsigned char*)malloc(q_bytes);
  unsigned char* o2 = (unsigned char*)malloc(q_bytes);
  if (!o1 || !o2) return 2;
  HIP_OK(hipMemcpy(o1, out1, q_bytes, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(o2, out2, q_bytes, hipMemcpyDeviceToHost));
  if (memcmp(o1, o2, q_bytes) != 0) {
    printf("FAIL the two streams' outputs differ\n");
    ++failures;
  } else {
    printf("ok outputs bitwise equal across streams\n");
  }
  snprintf(path, sizeof path, "%s/out.bin", dir);
  f = fopen(path, "wb");
  if (!f || fwrite(o1, 1, q_bytes, f) != q_bytes) {
    fprintf(stderr, "cannot write %s\n", path);
    return 2;
  }
  fclose(f);

  /* the same call captured into a graph and replayed: the workspace was
     reserved above, so the captured call allocates nothing */
  {
    hipGraph_t graph;
    hipGraphExec_t exec;
    HIP_OK(hipStreamBeginCapture(st, hipStreamCaptureModeGlobal));
    const int rc = paged_decode_attention(q, k, v, bt, lens, out2, batch, hq, hkv, d, page, num_pages, maxp, scale,
                                          st);
    HIP_OK(hipStreamEndCapture(st, &graph));
    expect("attention captured in a graph", rc, PDA_OK);
    HIP_OK(hipGraphInstantiate(&exec, graph, NULL, NULL, 0));
    for (int rep = 0; rep < 3; ++rep) {
      HIP_OK(hipMemset(out2, 0xFF, q_bytes));
      HIP_OK(hipGraphLaunch(exec, st));
      HIP_OK(hipStreamSynchronize(st));
      HIP_OK(hipMemcpy(o2, out2, q_bytes, hipMemcpyDeviceToHost));
      if (memcmp(o1, o2, q_bytes) != 0) {
        printf("FAIL graph replay %d differs from the eager call\n", rep);
        ++failures;
      }
    }
    if (failures == 0) printf("ok graph replays bitwise equal\n");
    HIP_OK(hipGraphExecDestroy(exec));
    HIP_OK(hipGraphDestroy(graph));
  }

  expect("release workspaces", pda_release_workspaces(), PDA_OK);
  HIP_OK(hipStreamDestroy(st));
  HIP_OK(hipFree(q));
  HIP_OK(hipFree(k));
  HIP_OK(hipFree(v));
  HIP_OK(hipFree(bt));
  HIP_OK(hipFree(lens));
  HIP_OK(hipFree(out1));
  HIP_OK(hipFree(out2));
  free(hq_);
  free(hk);
  free(hv);
  free(hbt);
  free(hlens);
  free(o1);
  free(o2);
  return failures ? 1 : 0;
}

int main(int argc, char** argv) {
  if (argc == 2 && strcmp(argv[1], "errors") == 0) return run_errors();
  if (argc == 3 && strcmp(argv[1], "run") == 0) return run_device(argv[2]);
  fprintf(stderr, "usage: %s errors | run DIR\n", argv[0]);
  return 2;
}
