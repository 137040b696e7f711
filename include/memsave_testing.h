/*
 * memsave_testing.h -- test hooks of libmemsave (not for production use).
 */
#ifndef MEMSAVE_TESTING_H
#define MEMSAVE_TESTING_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Make the next `n` transient-workspace allocations fail with MS_E_NOMEM,
 * so tests can check that a failed backward launches nothing, keeps its
 * record unconsumed and leaves the ledger unchanged. */
void ms_testing_fail_next_workspace(int32_t n);

/* Number of records currently allocated (leak check). */
int64_t ms_testing_live_records(void);

#ifdef __cplusplus
}
#endif

#endif /* MEMSAVE_TESTING_H */
