/* A plain C program that uses the library through include/mma.h alone: no
 * Python, no torch. It copies a ragged buffer host -> device -> host on its
 * own non-blocking stream, loads a three-tensor list, reads the stats, fetches
 * paged-KV blocks into buffers sized with mma_kv_layout_sizes, and checks every
 * byte against the source (a copy's and the KV layout's definition). The library is
 * initialised from the environment (MMA_* variables), so the same program
 * runs under either control mode. Prints "ALL OK" and exits 0 on success.
 */
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "mma.h"

static int failures = 0;

#define CHECK_MMA(call)                                                                       \
  do {                                                                                        \
    mma_status_t s_ = (call);                                                                 \
    if (s_ != MMA_OK) {                                                                       \
      printf("FAIL %s: %s (%s)\n", #call, mma_status_str(s_), mma_last_error());             \
      return 1;                                                                               \
    }                                                                                         \
  } while (0)

#define CHECK_HIP(call)                                                                       \
  do {                                                                                        \
    hipError_t e_ = (call);                                                                   \
    if (e_ != hipSuccess) {                                                                   \
      printf("FAIL %s: %s\n", #call, hipGetErrorString(e_));                                  \
      return 1;                                                                               \
    }                                                                                         \
  } while (0)

static void expect(int ok, const char* what) {
  if (!ok) {
    printf("FAIL %s\n", what);
    ++failures;
  }
}

int main(void) {
  const uint64_t n = (96u << 20) + 12345; /* several micro-tasks and a ragged tail */
  uint8_t *src = NULL, *back = NULL;
  void* dev = NULL;
  hipStream_t stream;
  mma_stats_t st;
  mma_config_t cfg;
  uint64_t i;

  CHECK_MMA(mma_init(0, NULL));
  CHECK_MMA(mma_get_config(&cfg));
  printf("control %u, chunk %llu, paths h2d 0x%x\n", cfg.control, (unsigned long long)cfg.chunk_bytes,
         cfg.path_mask_h2d);
  CHECK_MMA(mma_host_alloc(n, (void**)&src));
  CHECK_MMA(mma_host_alloc(n, (void**)&back));
  CHECK_HIP(hipMalloc(&dev, n));
  CHECK_HIP(hipStreamCreateWithFlags(&stream, hipStreamNonBlocking));
  for (i = 0; i < n; ++i) src[i] = (uint8_t)(i * 2654435761u >> 13);
  memset(back, 0xFF, n);

  /* host -> device -> host on one stream: stream order makes the second copy see the first */
  CHECK_MMA(mma_memcpy_async(dev, src, n, MMA_H2D, stream));
  CHECK_MMA(mma_memcpy_async(back, dev, n, MMA_D2H, stream));
  CHECK_HIP(hipStreamSynchronize(stream));
  expect(memcmp(back, src, n) == 0, "round trip differs from the source");

  /* a tensor list into three device tensors, then back with the blocking copy */
  {
    const uint64_t sz[3] = {5, 3u << 20, (17u << 20) + 3};
    void* d[3] = {NULL, NULL, NULL};
    mma_copy_desc_t list[3];
    uint64_t off = 0;
    int k;
    for (k = 0; k < 3; ++k) {
      CHECK_HIP(hipMalloc(&d[k], sz[k]));
      list[k].dst = d[k];
      list[k].src = src + off;
      list[k].bytes = sz[k];
      off += sz[k] + 4096;
    }
    CHECK_MMA(mma_weights_load(list, 3, MMA_H2D, stream));
    CHECK_HIP(hipStreamSynchronize(stream));
    off = 0;
    for (k = 0; k < 3; ++k) {
      memset(back, 0xFF, sz[k]);
      CHECK_MMA(mma_memcpy(back, d[k], sz[k], MMA_D2H));
      expect(memcmp(back, src + off, sz[k]) == 0, "tensor list entry differs from its source");
      off += sz[k] + 4096;
      CHECK_HIP(hipFree(d[k]));
    }
  }

  /* argument validation: pageable memory and a bad direction are rejected, nothing enqueued */
  {
    uint8_t* pageable = (uint8_t*)malloc(4096);
    expect(mma_memcpy_async(dev, pageable, 4096, MMA_H2D, stream) == MMA_ERR_NOT_PINNED,
           "pageable source accepted");
    expect(mma_memcpy_async(dev, src, 4096, 7, stream) == MMA_ERR_INVALID_ARG, "bad direction accepted");
    free(pageable);
  }

  CHECK_MMA(mma_synchronize(10000));
  CHECK_MMA(mma_get_stats(&st));
  {
    uint64_t total = 0;
    int p;
    for (p = 0; p < MMA_NUM_PATHS; ++p) total += st.path_bytes[p];
    printf("transfers %llu, failed %llu, bytes %llu (cu %llu)\n", (unsigned long long)st.transfers,
           (unsigned long long)st.failed_transfers, (unsigned long long)total,
           (unsigned long long)st.path_bytes[MMA_NUM_PATHS - 1]);
    expect(st.failed_transfers == 0, "a transfer failed");
    expect(st.transfers == 6, "transfer count");
    expect(total == 2 * n + 2 * ((3u << 20) + (17u << 20) + 8), "payload bytes");
  }
  /* a paged-KV fetch, its buffers sized with mma_kv_layout_sizes: every piece of every moved
   * block must equal its slot's piece in the pool (the layout's definition), the other GPU
   * blocks keep their fill */
  {
    mma_kv_layout_t lay = {2, 16, 2, 64, 2, 10, 8, MMA_KV_LAYOUT_PIECE};
    const int32_t slots[5] = {3, 0, 7, 5, 1}, blocks[5] = {9, 2, 4, 0, 6};
    uint64_t piece = 0, slot = 0, pool_bytes = 0, layer_bytes = 0;
    uint8_t *pool = NULL, *layer_host = NULL;
    void* layers[2] = {NULL, NULL};
    uint32_t l, k, j, b;
    mma_kv_layout_t wrap = {256, 1u << 16, 1u << 16, 1, 1, 1, 1u << 23, MMA_KV_LAYOUT_PIECE};
    expect(mma_kv_layout_sizes(&wrap, NULL, NULL, &pool_bytes, NULL) == MMA_ERR_INVALID_ARG,
           "a layout whose pool size wraps 64 bits was accepted");
    CHECK_MMA(mma_kv_layout_sizes(&lay, &piece, &slot, &pool_bytes, &layer_bytes));
    expect(piece == 4096 && slot == 4 * 4096 && pool_bytes == 8 * slot && layer_bytes == 2 * 10 * 4096,
           "layout sizes");
    CHECK_MMA(mma_host_alloc(pool_bytes, (void**)&pool));
    layer_host = (uint8_t*)malloc(layer_bytes);
    for (i = 0; i < pool_bytes; ++i) pool[i] = (uint8_t)(i * 40503u >> 7);
    for (l = 0; l < 2; ++l) {
      CHECK_HIP(hipMalloc(&layers[l], layer_bytes));
      CHECK_HIP(hipMemset(layers[l], 0x5A, layer_bytes));
    }
    CHECK_HIP(hipDeviceSynchronize());
    CHECK_MMA(mma_kv_fetch(&lay, pool, layers, slots, blocks, 5, stream));
    CHECK_HIP(hipStreamSynchronize(stream));
    for (l = 0; l < 2; ++l) {
      CHECK_HIP(hipMemcpy(layer_host, layers[l], layer_bytes, hipMemcpyDeviceToHost));
      for (k = 0; k < 2; ++k)
        for (b = 0; b < 10; ++b) {
          const uint8_t* got = layer_host + (k * 10 + b) * piece;
          int moved = -1;
          for (j = 0; j < 5; ++j)
            if ((uint32_t)blocks[j] == b) moved = (int)j;
          if (moved >= 0) {
            expect(memcmp(got, pool + slots[moved] * slot + (2 * l + k) * piece, piece) == 0,
                   "fetched KV piece differs from its pool slot");
          } else {
            for (i = 0; i < piece; ++i)
              if (got[i] != 0x5A) break;
            expect(i == piece, "a GPU block outside the table was written");
          }
        }
      CHECK_HIP(hipFree(layers[l]));
    }
    free(layer_host);
    CHECK_MMA(mma_host_free(pool));
  }

  CHECK_HIP(hipStreamDestroy(stream));
  CHECK_HIP(hipFree(dev));
  CHECK_MMA(mma_host_free(src));
  CHECK_MMA(mma_host_free(back));
  CHECK_MMA(mma_finalize());
  if (failures) {
    printf("FAILED: %d check(s)\n", failures);
    return 1;
  }
  printf("ALL OK\n");
  return 0;
}
