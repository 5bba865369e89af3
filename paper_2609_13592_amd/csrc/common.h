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

// Failure injection for host-memory allocation: true while the environment
// variable BOOST_FAULT_HOST_ALLOC is set to a non-zero integer.  Every
// allocation of host memory that backs pages (pinned host slabs) or a KV
// pool's allocator state then fails with BOOST_ENOMEM, so the failure path
// (release of everything allocated before, no partial object) can be tested
// without exhausting the machine.  Read at each such allocation (load time
// only, never on a decode call).
bool fault_host_alloc();

}  // namespace bst
