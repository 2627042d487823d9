// Host build of the trace-offset clamp the attention kernels apply to device
// cu_seqlens: for every offset pair, the trace the kernels address lies inside
// [0, ntok), is no longer than max_seqlen, and equals the given trace when the
// offsets are valid.  Prints "ok" and exits 0, or names the first failure.
#include <cstdio>

#include "kvs_device.h"

int main() {
  const int ntok = 1000;
  const int vals[] = {-2147483647 - 1, -5, -1, 0, 1, 7, 499, 500, 999, 1000, 1001, 5000, 2147483647};
  const int maxlens[] = {1, 64, 500, 1000, 4096};
  long checked = 0;
  for (int a : vals)
    for (int z : vals)
      for (int T : maxlens) {
        const kvs::Trace t = kvs::clamp_trace(a, z, ntok, T);
        const bool inside = t.tok0 >= 0 && t.L >= 0 && t.L <= T && (long)t.tok0 + t.L <= ntok;
        if (!inside) {
          std::printf("out of bounds: a=%d z=%d T=%d -> tok0=%d L=%d\n", a, z, T, t.tok0, t.L);
          return 1;
        }
        const bool valid = 0 <= a && a <= z && z <= ntok && z - a <= T;
        if (valid && (t.tok0 != a || t.L != z - a)) {
          std::printf("valid trace changed: a=%d z=%d T=%d -> tok0=%d L=%d\n", a, z, T, t.tok0, t.L);
          return 1;
        }
        ++checked;
      }
  // class switches: EMPTY -> PARTIAL, FULL -> PARTIAL, nothing else moves
  for (int c = 0; c < 3; ++c)
    for (int f = 0; f < 4; ++f) {
      int want = c;
      if ((f & 1) && c == kvs::kEmpty) want = kvs::kPartial;
      if ((f & 2) && c == kvs::kFull) want = kvs::kPartial;
      if (kvs::adjust_class(c, f) != want) {
        std::printf("adjust_class(%d, %d) = %d\n", c, f, kvs::adjust_class(c, f));
        return 1;
      }
    }
  std::printf("ok %ld\n", checked);
  return 0;
}
