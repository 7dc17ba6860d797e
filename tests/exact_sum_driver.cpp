// Host driver for exact_sum_f32 (paper_2608_21952_amd/csrc/exact_sum.hpp): reads a count n and
// n fp32 values (binary, native order) from stdin and writes the n prefix sums (fp64, binary).
#include <cstdint>
#include <cstdio>
#include <vector>

#include "exact_sum.hpp"

int main() {
  int32_t n = 0;
  if (std::fread(&n, sizeof n, 1, stdin) != 1 || n < 0) return 2;
  std::vector<float> v(n);
  if (n && std::fread(v.data(), sizeof(float), n, stdin) != (size_t)n) return 2;
  std::vector<double> out(n);
  for (int i = 0; i < n; ++i) out[i] = ssdi8::exact_sum_f32(v.data(), i + 1);
  if (n && std::fwrite(out.data(), sizeof(double), n, stdout) != (size_t)n) return 3;
  return 0;
}
