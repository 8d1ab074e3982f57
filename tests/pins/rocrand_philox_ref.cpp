// Test-only black-box reference: rocRAND's host-callable Philox4x32-10.
//
// Reads from stdin a mode word and a count n, then n records of three uint64
// values, and writes n results to stdout:
//   mode 1: record (seed, subsequence, offset) -> one uint32: the first rocrand()
//           after rocrand_init(seed, subsequence, offset).
//   mode 4: record (seed, subsequence, block)  -> four uint32: rocrand4() after
//           rocrand_init(seed, subsequence, 4 * block), i.e. one whole block.
// Neither the oracle nor the GPU library includes rocRAND; only this pin does.
#include <rocrand/rocrand_philox4x32_10.h>

#include <cstdint>
#include <cstdio>
#include <vector>

int main() {
  uint64_t head[2];
  if (std::fread(head, sizeof(uint64_t), 2, stdin) != 2) return 1;
  const uint64_t mode = head[0], n = head[1];
  std::vector<uint64_t> rec(3 * n);
  if (n && std::fread(rec.data(), sizeof(uint64_t), 3 * n, stdin) != 3 * n) return 1;
  std::vector<uint32_t> out;
  out.reserve(n * (mode == 4 ? 4 : 1));
  for (uint64_t i = 0; i < n; ++i) {
    rocrand_state_philox4x32_10 st;
    if (mode == 1) {
      rocrand_init(rec[3 * i], rec[3 * i + 1], rec[3 * i + 2], &st);
      out.push_back(rocrand(&st));
    } else {
      rocrand_init(rec[3 * i], rec[3 * i + 1], 4 * rec[3 * i + 2], &st);
      const uint4 v = rocrand4(&st);
      out.push_back(v.x); out.push_back(v.y); out.push_back(v.z); out.push_back(v.w);
    }
  }
  if (!out.empty()) std::fwrite(out.data(), sizeof(uint32_t), out.size(), stdout);
  return 0;
}
