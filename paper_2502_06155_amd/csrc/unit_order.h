// Order of the units within one XCD's share of a forward launch, shared by the
// kernel (device code) and the host-only schedule check: plain C++17 constexpr
// arithmetic, which hipcc also compiles for the device.
#pragma once

#include <stdint.h>

namespace ta {

// Units of XCD x when n units are dealt out to the 8 XCDs as contiguous shares:
// XCD x owns [share_start(n, x), share_start(n, x) + share_count(n, x)).
constexpr uint32_t share_count(uint32_t n, uint32_t x) { return n / 8 + (x < n % 8 ? 1u : 0u); }
constexpr uint32_t share_start(uint32_t n, uint32_t x) { return x * (n / 8) + (x < n % 8 ? x : n % 8); }

// The unit that queue position pos of XCD x runs when every segment of the launch
// ends on a short query block (nqb > 1 blocks per segment, unit u = s * nqb + qb with
// the short block at qb = nqb - 1): the share's full blocks first, in their order,
// then its short blocks, in theirs. A short block finishes in about half the time of
// a full one; run among them, it would let the next unit of the share start early
// and out of step with the other blocks of its segment, which then no longer stream
// the same K/V tiles through L2 together.
constexpr uint32_t short_last_unit(uint32_t n, uint32_t nqb, uint32_t x, uint32_t pos) {
  const uint32_t s = share_start(n, x), e = s + share_count(n, x);
  const uint32_t f0 = s - s / nqb;                 // full blocks of the launch before s
  const uint32_t n_full = (e - e / nqb) - f0;      // full blocks in the share
  if (pos < n_full) {
    const uint32_t j = f0 + pos;                   // the j-th full block of the launch
    return j / (nqb - 1) * nqb + j % (nqb - 1);
  }
  return (s / nqb + (pos - n_full)) * nqb + nqb - 1;  // short blocks from s on
}

}  // namespace ta
