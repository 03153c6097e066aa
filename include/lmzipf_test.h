/*
 * lmzipf_test.h — test-only entry points of liblmzipf.so. Not part of the
 * training interface declared in lmzipf.h: nothing on the hot path calls
 * these, and a trainer never should.
 */
#ifndef LMZIPF_TEST_H
#define LMZIPF_TEST_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Forces the failure path of the bounded waits between workgroups, so that
 * tests can check it from the host without any kernel hanging. While enable
 * is nonzero, the fix-up workgroups of lm_segsum's one-launch form wait for
 * a flag value that the walk never writes, and the look-backs of lm_unique's
 * multi-workgroup kernels (inputs above 8,192 ids) read every predecessor as
 * not ready: each such wait gives up after spin_limit polls (at least 1) and
 * sets LM_DEVERR_SPIN in dev_err. The launches still finish and write only
 * inside their buffers; their results are then unspecified. Process-wide;
 * off by default. Returns LM_OK (0). */
int lm_test_force_wait_failure(int32_t enable, uint32_t spin_limit);

#ifdef __cplusplus
}
#endif

#endif /* LMZIPF_TEST_H */
