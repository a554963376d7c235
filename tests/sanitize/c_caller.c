/* Calls into the library as a C program does: in C an enum argument is an
 * int, and any int value may be passed.  Used by host_driver.cpp for the
 * out-of-range enum values it may not form itself in C++.  Also checks that
 * the public header compiles as C. */
#include <stdint.h>

#include "na.h"

int c_validate(int rank, const int64_t* L, const int32_t* k, const int32_t* d, int64_t B,
               int64_t H, int64_t D, int dtype) {
    return (int)na_validate(rank, L, k, d, NULL, B, H, D, (na_dtype)dtype, 1.0f);
}

int c_forward(int rank, const int64_t* L, const int32_t* k, const int32_t* d, int64_t B,
              int64_t H, int64_t D, int dtype, void* buf) {
    return (int)na_forward(rank, L, k, d, NULL, B, H, D, (na_dtype)dtype, 1.0f, buf, buf, buf, buf,
                           (float*)buf, NULL);
}

int c_candidates(int rank, const int64_t* L, const int32_t* k, const int32_t* d, int64_t B,
                 int64_t H, int64_t D, int dtype) {
    return na_candidate_tilings(rank, L, k, d, B, H, D, (na_dtype)dtype, 1, NULL, 0);
}

int c_unfused_softmax(int rank, const int64_t* L, const int32_t* k, const int32_t* d, int64_t B,
                      int64_t H, int64_t D, int dtype, void* buf) {
    return (int)na_unfused_softmax(rank, L, k, d, NULL, B, H, D, (na_dtype)dtype, buf, (float*)buf,
                                   NULL);
}

const char* c_status_string(int status) { return na_status_string((na_status)status); }
