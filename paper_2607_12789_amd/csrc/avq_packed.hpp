// Packed aggregates: what the aggregation writes for the attention kernel.
//
// Codes are grouped in octets of 8. Per (batch, head) the buffer holds
//   means  [n_oct][d][8]  dtype   the mean value Vbar/n of every code of the
//                                 octet (slot s = code s of the octet), 0 for
//                                 empty codes and padding slots;
//   info   [n_oct][16]    fp32    slots 0..7: n of each code (as a float),
//                                 slots 8..15: ln n (-inf for n = 0 and
//                                 padding).
// Octet order: the parent octets (parents 8o .. 8o+7), padded with empty
// octets to a multiple of 8 octets (64 parents, one attention chunk); then,
// for every parent p, its ceil(Ch/8) child octets (children 8j .. 8j+7, slots
// past Ch empty); then one empty octet (all means 0, n 0, ln n -inf).
//
// The mean octet [d][8] is exactly the A operand of the value product for one
// lane: 8 consecutive codes of one column d.
#pragma once

#include <stddef.h>

namespace avq {

struct PackedLayout {
  int PO;            // parent octets (a multiple of 8)
  int CO;            // child octets per parent
  int n_oct;         // all octets, the empty one included
  int zero_oct;      // index of the empty octet
  size_t oct_bytes;  // bytes of one mean octet
  size_t info_off;   // byte offset of the info section
  size_t bytes;      // bytes per (batch, head)
};

__host__ __device__ inline PackedLayout packed_layout(int M0, int Ch, int d, int esize) {
  PackedLayout L;
  L.PO = ((M0 + 63) / 64) * 8;
  L.CO = (Ch + 7) / 8;
  L.n_oct = L.PO + M0 * L.CO + 1;
  L.zero_oct = L.n_oct - 1;
  L.oct_bytes = (size_t)8 * d * esize;
  L.info_off = (size_t)L.n_oct * L.oct_bytes;
  L.bytes = L.info_off + (size_t)L.n_oct * 16 * sizeof(float);
  return L;
}

}  // namespace avq
