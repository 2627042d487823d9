// Host build of the tile-copy addressing (RowStager) of every staged tile the
// kernels use.  For trace tails of every length and several row strides:
//  * every LDS slot of the tile is written exactly once, by one lane of one
//    piece of one wave, and no slot past the tile;
//  * every source read (16 bytes) lies inside rows row0 .. rmax of the tensor;
//  * a slot of a row inside the trace receives that row's data chunk, and each
//    16-byte data chunk of such a row lands in exactly one slot (the swizzle
//    is a permutation), so the padded tile holds the rows unchanged.
// Prints "ok" and exits 0, or names the first failure.
#include <cstdio>
#include <vector>

#include "kvs_device.h"

template <int D, int R, int NW, bool COMPACT>
static int check(const char* name) {
  using ST = kvs::RowStager<D, R, NW, COMPACT>;
  using LY = kvs::Lay<D, COMPACT>;
  const long long strides[] = {D, 2LL * D, 8LL * D, 40LL * D};
  long checked = 0;
  for (long long stride : strides)
    for (int dr = 0; dr < R + 3; ++dr) {   // dr = rmax - row0: last valid row of the tile
      const uint32_t lim = ST::limit(dr, stride);
      std::vector<int> written(ST::NI * kvs::kWave + kvs::kWave, 0);
      std::vector<int> chunk_seen(R * LY::CPR, 0);
      for (int wave = 0; wave < NW; ++wave)
        for (int i = 0; i < ST::PW; ++i) {
          const int n = wave + i * NW;
          if (!ST::issues(i, n)) continue;
          if (n >= ST::NI) {
            std::printf("%s: wave %d piece %d issues slot group %d past the tile\n", name, wave, i, n);
            return 1;
          }
          for (int lane = 0; lane < kvs::kWave; ++lane) {
            ++written[n * kvs::kWave + lane];
            const uint32_t off = ST::src_offset(n, lane, stride);
            const uint32_t src = off < lim ? off : lim;
            const long long end = (long long)src + 16;
            const long long hi = ((long long)(dr < R - 1 ? dr : R - 1) * stride + D) * 2;
            if (end > hi) {
              std::printf("%s: stride %lld dr %d wave %d piece %d lane %d reads [%u, %lld) past %lld\n", name,
                          stride, dr, wave, i, lane, src, end, hi);
              return 1;
            }
            int r, col;
            ST::slot(n, lane, r, col);
            const int pc = n * kvs::kWave + lane - r * LY::CPRP;
            if (r <= dr && pc < LY::CPR) {
              if (src != (uint32_t)(r * stride + col) * 2u) {
                std::printf("%s: row %d inside the trace moved (stride %lld dr %d)\n", name, r, stride, dr);
                return 1;
              }
              if (LY::off(r, col) != r * LY::PITCH + 8 * pc) {
                std::printf("%s: slot of row %d chunk %d does not hold column %d\n", name, r, pc, col);
                return 1;
              }
              ++chunk_seen[r * LY::CPR + col / 8];
            }
            ++checked;
          }
        }
      for (int q = 0; q < (int)written.size(); ++q) {
        const int want = q < ST::NI * kvs::kWave ? 1 : 0;
        if (written[q] != want) {
          std::printf("%s: slot %d written %d times\n", name, q, written[q]);
          return 1;
        }
      }
      for (int r = 0; r < R && r <= dr; ++r)
        for (int c = 0; c < LY::CPR; ++c)
          if (chunk_seen[r * LY::CPR + c] != 1) {
            std::printf("%s: row %d chunk %d staged %d times\n", name, r, c, chunk_seen[r * LY::CPR + c]);
            return 1;
          }
    }
  std::printf("%s: %ld lane copies checked\n", name, checked);
  return 0;
}

int main() {
  if (check<128, 32, 4, true>("forward K/V sub-tile, D=128")) return 1;
  if (check<64, 64, 4, true>("forward K/V tile, D=64")) return 1;
  if (check<128, 64, 4, true>("dQ K/V tile, D=128")) return 1;
  if (check<64, 64, 4, true>("dQ K/V tile, D=64")) return 1;
  if (check<128, 64, 8, false>("dK/dV Q/dO tile, D=128")) return 1;
  if (check<64, 64, 8, false>("dK/dV Q/dO tile, D=64")) return 1;
  std::printf("ok\n");
  return 0;
}
