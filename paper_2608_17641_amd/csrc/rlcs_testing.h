// Test-only entry point of librlcs.so, not part of the public interface in rlcs.h.
#pragma once

#include "rlcs.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Forces a kernel variant for the calls made afterwards FROM THE CALLING THREAD (the setting is
 * thread-local, so it never affects other threads' calls): 0 = automatic choice, 1 = whole rows
 * per workgroup (and, for whitened masked GAE, the two-pass whitening), 2 = rows split across
 * workgroups (needs the workspace; calls of more than 1024 rows, or columns in more than 1024
 * blocks of 64, still run whole), 3 = column scans in narrow
 * groups (16 float32 or 32 bfloat16 columns per workgroup, whole columns; row-major calls as
 * with 0), 4 = column scans in narrow groups split across workgroups along T, the tiles drawn
 * in arrival order (needs the workspace; at most 1024 groups and more than 64 steps, else as
 * with 0; row-major calls as with 0). Returns RLCS_ERR_INVALID_ARG for other values. */
rlcs_status rlcs_testing_set_variant(int variant);

#ifdef __cplusplus
}
#endif
