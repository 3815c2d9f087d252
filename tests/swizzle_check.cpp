// Host-side check of the LDS unit layout shared by the bf16 expert GEMMs
// (lds_dma.h): DMA lane i of a unit lands at byte 16 i (row i / 8, slot i % 8)
// holding chunk unit_chunk(i) of its row; every 8 lanes fetch their row's 8
// chunks exactly once (whole cache lines), and the MFMA operand each lane reads
// from unit_read_offset(lane, h) is row lane % 16, k chunk 4 h + lane / 16 of the
// 16-row block (two units).  Prints "ok" and exits 0, else the first mismatch.
#include <cstdio>

#include "../paper_2609_05228_amd/csrc/lds_dma.h"

int main() {
  for (int row = 0; row < 8; ++row) {
    int seen = 0;
    for (int s = 0; s < 8; ++s) seen |= 1 << ace::unit_chunk(row * 8 + s);
    if (seen != 0xFF) {
      std::printf("row %d: DMA lanes do not fetch each chunk once (mask %x)\n", row, seen);
      return 1;
    }
  }
  for (int h = 0; h < 2; ++h)
    for (int lane = 0; lane < 64; ++lane) {
      const int off = ace::unit_read_offset(lane, h);
      if (off < 0 || off >= 2 * ace::kUnitBytes || off % 16) {
        std::printf("lane %d h %d: offset %d outside the block\n", lane, h, off);
        return 1;
      }
      const int unit = off / ace::kUnitBytes, line = (off % ace::kUnitBytes) / 128, slot = (off % 128) / 16;
      const int row = unit * 8 + line, chunk = ace::unit_chunk(line * 8 + slot);
      if (row != (lane & 15) || chunk != 4 * h + (lane >> 4)) {
        std::printf("lane %d h %d: reads row %d chunk %d, wants row %d chunk %d\n", lane, h, row, chunk, lane & 15,
                    4 * h + (lane >> 4));
        return 1;
      }
    }
  std::printf("ok\n");
  return 0;
}
