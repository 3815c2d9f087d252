// Host-side check of the grouped GEMM's wait counts (gemm_pipe.h): for every tile
// shape the kernels instantiate, every K length up to 128 stages and every per-wave
// activation DMA count, replay the wave's DMA issue sequence one instruction at a
// time and compare pending_ok with the count of DMAs issued after the later of
// A(kt) and B(kt) at the wait before stage kt (vmcnt completes in issue order),
// and the closed form (Closed) with it wherever the kernels use it.
// Also checks that both stages were issued before their wait, that the count fits
// the 0..63 wait table, and that a refilled ring slot held the stage consumed in
// the previous iteration.  Prints "ok" and exits 0, else the first mismatch.
#include <cstdio>
#include <vector>

#include "../paper_2609_05228_amd/csrc/gemm_pipe.h"

template <int MB, int CG, int KH, int W>
static bool check() {
  using P = ace::Pipe<MB, CG, KH, W>;
  for (int nk = 1; nk <= 128; ++nk)
    for (int na = 0; na <= P::NA_MAX; ++na) {
      std::vector<int> last_a(nk, -1), last_b(nk, -1);  // index of the last DMA of each stage
      int issued = 0;
      auto issue_a = [&](int s) { for (int i = 0; i < na; ++i) last_a[s] = issued++; };
      auto issue_b = [&](int s) { for (int i = 0; i < P::NB; ++i) last_b[s] = issued++; };
      for (int s = 0; s < P::SB - 1 && s < nk; ++s) issue_b(s);
      for (int s = 0; s < P::SA - 1 && s < nk; ++s) issue_a(s);
      for (int kt = 0; kt < nk; ++kt) {
        if (last_b[kt] < 0 || (na > 0 && last_a[kt] < 0)) {
          std::printf("MB=%d CG=%d KH=%d nk=%d na=%d: stage %d not issued before its wait\n", MB, CG, KH, nk, na, kt);
          return false;
        }
        const int end = (last_a[kt] > last_b[kt] ? last_a[kt] : last_b[kt]) + 1;
        const int want = issued - end;
        const int got = ace::pending_ok<P>(kt, nk, na);
        if (got != want || got < 0 || got > 63) {
          std::printf("MB=%d CG=%d KH=%d nk=%d na=%d kt=%d: pending_ok %d, replay %d\n", MB, CG, KH, nk, na, kt, got,
                      want);
          return false;
        }
        using CF = ace::Closed<P>;
        if (CF::on && na > 0 && want != (CF::nb_pending(kt, nk) ? P::NB : 0)) {
          std::printf("MB=%d CG=%d KH=%d nk=%d na=%d kt=%d: closed-form count %d, replay %d\n", MB, CG, KH, nk, na, kt,
                      CF::nb_pending(kt, nk) ? P::NB : 0, want);
          return false;
        }
        // slots refilled in this iteration held stage kt - 1 (consumed before the barrier)
        if (kt >= 1 && kt + P::SA - 1 < nk && ((kt + P::SA - 1) % P::SA) != ((kt - 1) % P::SA)) {
          std::printf("A slot reuse\n");
          return false;
        }
        if (kt >= 1 && kt + P::SB - 1 < nk && ((kt + P::SB - 1) % P::SB) != ((kt - 1) % P::SB)) {
          std::printf("B slot reuse\n");
          return false;
        }
        if (kt + P::SA - 1 < nk) issue_a(kt + P::SA - 1);
        if (kt + P::SB - 1 < nk) issue_b(kt + P::SB - 1);
      }
    }
  return true;
}

int main() {
  constexpr int W = 8;
  bool ok = check<4, 8, 2, W>() && check<8, 8, 2, W>() && check<12, 8, 2, W>() && check<16, 8, 2, W>() &&
            check<4, 4, 2, W>() && check<8, 4, 2, W>() && check<12, 4, 2, W>() && check<16, 4, 2, W>() &&
            check<4, 8, 1, W>() && check<16, 8, 1, W>() && check<16, 4, 1, W>();
  std::printf(ok ? "ok\n" : "FAILED\n");
  return ok ? 0 : 1;
}
