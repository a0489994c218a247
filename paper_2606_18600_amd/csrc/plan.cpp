// Host-side sizing rules shared by the launchers and the stage runtime: how
// many K ranges a split-K decode GEMM takes and how many positions one
// prefill attention work item covers. Plain host code (no HIP calls).
#include <algorithm>
#include <cstdlib>

#include "kernels.hpp"

namespace stage_k {

int skinny_kb_len(int K, int splits) {
  int kb = (K + splits - 1) / splits;
  return (kb + 63) / 64 * 64;
}

int skinny_splits(int N, int K, int target_blocks, int max_splits) {
  const int col_blocks = (N / 64 + kSkinnyWaves - 1) / kSkinnyWaves;
  int s = std::max(1, target_blocks / col_blocks);
  s = std::min(s, std::min(max_splits, K / 64));
  // the number of K ranges actually launched after rounding the range up
  const int kb = skinny_kb_len(K, s);
  return (K + kb - 1) / kb;
}

bool skinny_kp_enabled() {
  static const bool on = [] {
    const char* v = std::getenv("STAGE_SKINNY_KP");
    return !(v && *v && std::atoi(v) == 0);
  }();
  return on;
}

bool skinny_kp_used(int K, int splits, bool swiglu) {
  return !swiglu && splits > 1 && K % 128 == 0 && skinny_kp_enabled();
}

int skinny_kp_kb_len(int K, int splits) {
  int kb = (K + splits - 1) / splits;
  return (kb + 127) / 128 * 128;
}

int skinny_kp_splits(int N, int K, int target_blocks, int max_splits) {
  const int col_blocks = (N / 64 + kSkinnyKpGroups - 1) / kSkinnyKpGroups;
  int s = std::max(1, target_blocks / col_blocks);
  s = std::min(s, std::min(max_splits, K / 128));
  const int kb = skinny_kp_kb_len(K, s);
  return (K + kb - 1) / kb;
}

int prefill_item_positions(DType dt, int group) {
  (void)dt;
  return kPrefillRows / group;
}

}  // namespace stage_k
