// Host-side conversion of layer matrices from row-major to fragment order
// (the layout device.h's w16_index / w4_byte / w4_sm read): each 16-row
// block of a matrix is laid out so that one wave's load of an MFMA operand
// fragment is one contiguous 1 KiB read.  Row groups are split over threads.
#include <algorithm>
#include <cstring>
#include <system_error>
#include <thread>
#include <vector>

#include "pack.h"

namespace pipo {

void parallel_ranges(int64_t n, int64_t nt, const std::function<void(int64_t, int64_t)>& fn) {
  nt = std::max<int64_t>(1, std::min(nt, n));
  if (nt <= 1) {
    if (n > 0) fn(0, n);
    return;
  }
  std::vector<std::thread> th;
  th.reserve((size_t)nt);
  const int64_t per = (n + nt - 1) / nt;
  int64_t a = 0;
  for (; a < n; a += per) {
    try {
      th.emplace_back(fn, a, std::min(n, a + per));
    } catch (const std::system_error&) {
      break;
    }
  }
  if (a < n) fn(a, n);
  for (auto& t : th) t.join();
}

static void over_row_groups(int64_t groups, const std::function<void(int64_t, int64_t)>& fn) {
  parallel_ranges(groups,
                  std::min<int64_t>({16, (int64_t)std::thread::hardware_concurrency(),
                                     groups / 64 + 1}),
                  fn);
}

void pack_f16(const uint16_t* W, uint16_t* out, int64_t N, int64_t K) {
  // block (rg, kb) = 512 halves; lane slot r + 16 g holds row 16 rg + r, k = 32 kb + 8 g ..
  over_row_groups(N / 16, [=](int64_t g0, int64_t g1) {
    for (int64_t rg = g0; rg < g1; ++rg)
      for (int64_t kb = 0; kb < K / 32; ++kb) {
        uint16_t* blk = out + (rg * (K / 32) + kb) * 512;
        for (int g = 0; g < 4; ++g)
          for (int r = 0; r < 16; ++r)
            std::memcpy(blk + (r + 16 * g) * 8, W + (rg * 16 + r) * K + kb * 32 + g * 8, 16);
      }
  });
}

void pack_w4_codes(const uint8_t* q, uint8_t* out, int64_t N, int64_t K) {
  // block (rg, kb) = 1 KiB; lane slot r + 16 g holds row 16 rg + r's codes for k = 128 kb + 32 g ..
  over_row_groups(N / 16, [=](int64_t g0, int64_t g1) {
    for (int64_t rg = g0; rg < g1; ++rg)
      for (int64_t kb = 0; kb < K / 128; ++kb) {
        uint8_t* blk = out + (rg * (K / 128) + kb) * 1024;
        for (int g = 0; g < 4; ++g)
          for (int r = 0; r < 16; ++r)
            std::memcpy(blk + (r + 16 * g) * 16, q + (rg * 16 + r) * (K / 2) + kb * 64 + g * 16,
                        16);
      }
  });
}

void pack_w4_scale_min(const uint16_t* sm, uint16_t* out, int64_t N, int64_t K) {
  // per block (rg, kb) 32 pairs: row r's groups 2 kb, 2 kb + 1 at 2 r, 2 r + 1
  const uint32_t* in = reinterpret_cast<const uint32_t*>(sm);
  uint32_t* o = reinterpret_cast<uint32_t*>(out);
  over_row_groups(N / 16, [=](int64_t g0, int64_t g1) {
    for (int64_t rg = g0; rg < g1; ++rg)
      for (int64_t kb = 0; kb < K / 128; ++kb)
        for (int r = 0; r < 16; ++r)
          for (int j = 0; j < 2; ++j)
            o[(rg * (K / 128) + kb) * 32 + r * 2 + j] = in[(rg * 16 + r) * (K / 64) + kb * 2 + j];
  });
}

}  // namespace pipo

using namespace pipo;

extern "C" {

pipo_status pipo_pack_f16(const uint16_t* W, uint16_t* out, int64_t N, int64_t K) {
  clear_error();
  if (!W || !out || N <= 0 || K <= 0 || N % 16 != 0 || K % 32 != 0 || W == out) {
    set_error("pack_f16: NULL or aliased buffers, or N %% 16 / K %% 32 != 0");
    return PIPO_ERR_ARG;
  }
  return guarded([&] {
    pack_f16(W, out, N, K);
    return PIPO_OK;
  });
}

pipo_status pipo_pack_w4(const uint8_t* q, const uint16_t* scale_min, uint8_t* q_out,
                         uint16_t* scale_min_out, int64_t N, int64_t K) {
  clear_error();
  if (!q || !scale_min || !q_out || !scale_min_out || N <= 0 || K <= 0 || N % 16 != 0 ||
      K % 128 != 0 || (const void*)q == q_out || scale_min == scale_min_out) {
    set_error("pack_w4: NULL or aliased buffers, or N %% 16 / K %% 128 != 0");
    return PIPO_ERR_ARG;
  }
  return guarded([&] {
    pack_w4_codes(q, q_out, N, K);
    pack_w4_scale_min(scale_min, scale_min_out, N, K);
    return PIPO_OK;
  });
}

}  // extern "C"
