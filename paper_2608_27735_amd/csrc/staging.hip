// staging.hip -- upload of cached partition renders from pinned host memory
// (Method section: the cache of camera-partition renders lives off the GPU and
// the renders a camera needs are brought in when a block becomes active).
//
// Only each image's coverage box is copied, one 2D DMA per image (rows of the
// box, pitch = image row): the bytes over PCIe follow what the partition
// covers, not the frame size. The copies run on the caller's stream, so a
// caller can double-buffer them against the collapse of the previous chunk.
#include "abcd_internal.h"

namespace abcd {

int32_t stage_cached(int width, int height, int k, const uint16_t* const* host_images,
                     const int32_t* rects, uint16_t* dst, hipStream_t stream) {
  const size_t row = (size_t)width * 4 * sizeof(uint16_t);
  const size_t img = row * (size_t)height;
  for (int j = 0; j < k; ++j) {
    int x0 = 0, y0 = 0, x1 = width, y1 = height;
    if (rects) {
      x0 = rects[4 * j];
      y0 = rects[4 * j + 1];
      x1 = rects[4 * j + 2];
      y1 = rects[4 * j + 3];
    }
    if (x1 <= x0 || y1 <= y0) continue;
    const size_t off = (size_t)y0 * row + (size_t)x0 * 4 * sizeof(uint16_t);
    const char* src = reinterpret_cast<const char*>(host_images[j]) + off;
    char* d = reinterpret_cast<char*>(dst) + (size_t)j * img + off;
    const size_t wbytes = (size_t)(x1 - x0) * 4 * sizeof(uint16_t);
    ABCD_HIP(hipMemcpy2DAsync(d, row, src, row, wbytes, (size_t)(y1 - y0), hipMemcpyHostToDevice,
                              stream));
  }
  return ABCD_OK;
}

}  // namespace abcd
