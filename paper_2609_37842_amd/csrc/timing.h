// Optional per-kernel-class timing with HIP events (for measurement harnesses).
// When enabled, every launch of a timed class is bracketed by two events
// recorded on the launching stream; eogp_timing_read sums their elapsed times.
#pragma once
#include "common.h"

namespace eogp {
namespace timing {

bool enabled();
int begin(int cls, hipStream_t s);          // returns a slot id, or -1 when disabled
void end(int slot, hipStream_t s);

struct Scope {
  int slot;
  hipStream_t s;
  Scope(int cls, hipStream_t st) : slot(begin(cls, st)), s(st) {}
  ~Scope() { end(slot, s); }
};

}  // namespace timing
}  // namespace eogp
