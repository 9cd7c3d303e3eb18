// Interface of the CPU stand-ins for the HIP runtime and kernel launchers
// (fake_hip.cpp), used by the host-logic test program.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

struct FakeShape {
  int64_t tp = 0, tr = 0;
  std::vector<int32_t> cu_prompt, cu_resp;
};

struct FakeCounts {
  int64_t fwd_pairs = 0, dq_pairs = 0, dkv_pairs = 0;
  int launches = 0;
};

void fake_set_shape(const FakeShape& s);
void fake_fail_at(long n);
const FakeCounts& fake_counts();
const std::vector<std::string>& fake_errors();
void fake_check_coverage(const char* name, int64_t rows);
void fake_reset_coverage();
// the workspace of the call under test: row maps inside it are checked
void fake_set_workspace(const void* ws, size_t bytes);
// per fp32 slab row: how many dK/dV tiles wrote it
const std::vector<int>& fake_slab_rows();
