// Shared host-side helpers of the library: error reporting and constants.
#pragma once
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>
#include <vector>

#include "../../include/boost_cap.h"

namespace bst {

constexpr uint64_t kPage = BOOST_PAGE_BYTES;

// Record a message for boost_last_error() and return `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// C2 tier map of one tensor (modulo placement over superpages).
int mpp_tiers(uint64_t bytes, uint32_t M, uint64_t footprint,
              std::vector<uint8_t>& tiers);
uint64_t pages_of(uint64_t bytes);

}  // namespace bst
