// Host-side conversion of layer matrices to fragment order (pack.cpp).
#pragma once

#include <functional>

#include "common.h"

namespace pipo {

void pack_f16(const uint16_t* W, uint16_t* out, int64_t N, int64_t K);
void pack_w4_codes(const uint8_t* q, uint8_t* out, int64_t N, int64_t K);
void pack_w4_scale_min(const uint16_t* sm, uint16_t* out, int64_t N, int64_t K);

}  // namespace pipo
