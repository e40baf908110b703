// Host checks of the validate mode (block lists and sample offsets), run on
// the CPU against the library built with AddressSanitizer and
// UndefinedBehaviorSanitizer. Prints one line per case and exits non-zero on
// the first case whose status or message is not the expected one.
#include <cstdio>
#include <cstring>
#include <vector>

#include "common.h"

namespace {
int failures = 0;

void expect(const char* name, ut_status got, ut_status want, const char* needle) {
  const char* msg = ut_last_error();
  const bool ok = got == want && (want == UT_OK || std::strstr(msg, needle) != nullptr);
  std::printf("%-44s %s (status %d, \"%s\")\n", name, ok ? "ok" : "FAIL", (int)got, msg);
  if (!ok) ++failures;
}
}  // namespace

int main() {
  using ut::check_cu_seqlens;
  using ut::check_lists;
  // 3 rows over 5 columns: {0, 2}, {}, {1, 3, 4}
  std::vector<int32_t> ptr = {0, 2, 2, 5}, idx = {0, 2, 1, 3, 4};
  expect("lists: well formed", check_lists("t", "rows", ptr.data(), idx.data(), 5, 3, 5), UT_OK, "");
  expect("lists: pointers only", check_lists("t", "rows", ptr.data(), nullptr, 0, 3, 5), UT_OK, "");
  std::vector<int32_t> p1 = {1, 2, 2, 5};
  expect("lists: start not 0", check_lists("t", "rows", p1.data(), idx.data(), 5, 3, 5),
         UT_ERR_INVALID_ARG, "start at 1");
  std::vector<int32_t> p2 = {0, 3, 2, 5};
  expect("lists: decreasing pointers", check_lists("t", "rows", p2.data(), idx.data(), 5, 3, 5),
         UT_ERR_INVALID_ARG, "decrease at row 1");
  expect("lists: end past the entries", check_lists("t", "rows", ptr.data(), idx.data(), 4, 3, 5),
         UT_ERR_INVALID_ARG, "pointers end at 5");
  std::vector<int32_t> i1 = {0, 2, 1, 3, 5};
  expect("lists: entry out of range", check_lists("t", "rows", ptr.data(), i1.data(), 5, 3, 5),
         UT_ERR_INVALID_ARG, "holds 5");
  std::vector<int32_t> i2 = {0, 2, 1, -1, 4};
  expect("lists: negative entry", check_lists("t", "rows", ptr.data(), i2.data(), 5, 3, 5),
         UT_ERR_INVALID_ARG, "holds -1");
  std::vector<int32_t> i3 = {2, 2, 1, 3, 4};
  expect("lists: repeated entry", check_lists("t", "rows", ptr.data(), i3.data(), 5, 3, 5),
         UT_ERR_INVALID_ARG, "not strictly ascending");
  std::vector<int32_t> i4 = {0, 2, 3, 1, 4};
  expect("lists: descending entry", check_lists("t", "rows", ptr.data(), i4.data(), 5, 3, 5),
         UT_ERR_INVALID_ARG, "row 2 is not strictly ascending");
  std::vector<int32_t> empty_ptr = {0, 0, 0};
  expect("lists: all rows empty", check_lists("t", "rows", empty_ptr.data(), nullptr, 0, 2, 5),
         UT_OK, "");

  std::vector<int32_t> cu = {0, 100, 100, 250};
  expect("cu_seqlens: well formed (empty sample)", check_cu_seqlens("t", cu.data(), 3, 250, 150), UT_OK, "");
  expect("cu_seqlens: wrong total", check_cu_seqlens("t", cu.data(), 3, 251, 150),
         UT_ERR_INVALID_ARG, "from 0 to T = 251");
  std::vector<int32_t> c2 = {0, 120, 100, 250};
  expect("cu_seqlens: decreasing", check_cu_seqlens("t", c2.data(), 3, 250, 200),
         UT_ERR_INVALID_ARG, "decreases at sample 1");
  expect("cu_seqlens: sample over max_seqlen", check_cu_seqlens("t", cu.data(), 3, 250, 149),
         UT_ERR_INVALID_ARG, "sample 2 has 150 tokens");
  std::printf("%d failure(s)\n", failures);
  return failures != 0;
}
