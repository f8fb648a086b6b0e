// Kernel timing instrumentation (fo_profile_enable / fo_profile_read).
#pragma once

#include "common.h"

namespace fo {

enum ProfKind : int { PROF_GEMM = 0, PROF_ATTN_FWD = 1, PROF_ATTN_BWD = 2, PROF_OTHER = 3 };

struct ProfInfo {
    int kind = PROF_OTHER;
    // GEMM: algorithmic flops 2*M*N*K with M, K taken from *Mdev / *Kdev when set
    int M = 0, N = 0, K = 0, nseg = 1;
    // grouped GEMM launch: ngroup products, their N; the kernel snapshots (M, K) of each
    int ngroup = 0;
    int gN[4] = {0, 0, 0, 0};
    const int* Mdev = nullptr;
    const int* Kdev = nullptr;
    // attention: cu[B+1] packed offsets, width d
    const int* cu = nullptr;
    int B = 0, d = 0;
};

// Returns a record handle (>= 0) when the calling thread is profiling, else -1.
// Call before the launch; prof_end after it, on the same stream.  When the
// launch has device-side sizes, the kernel copies them into prof_snap(h)
// (GEMM: effective M and K; attention: cu[0..B]) from its first workgroup.
int prof_begin(hipStream_t s, const char* name, const ProfInfo& info);
void prof_end(int h, hipStream_t s);
// The same record for a launch through hipExtLaunchKernelGGL, which stamps the
// returned start / stop events at the kernel's own dispatch begin and end (no
// event packets around it): *a = *b = nullptr when the thread is not profiling.
int prof_begin_ext(const char* name, const ProfInfo& info, hipEvent_t* a, hipEvent_t* b);
void prof_end_ext(int h);
int* prof_snap(int h);  // NULL when h < 0
bool prof_active();     // the calling thread is recording launches
constexpr int kProfSnapInts = 258;  // capacity of one snapshot (cu of up to 257 offsets)

}  // namespace fo
