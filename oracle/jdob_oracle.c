/*
 * jdob_oracle.c — CPU oracle for batched J-DOB, binary32 and binary64.
 * TEST INFRASTRUCTURE ONLY (see jdob_oracle.h).  Build with
 * -ffp-contract=off and without fast-math: the decisions must come from the
 * exact IEEE operation sequence written in jdob_oracle_body.h.
 */
#include "jdob_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#if defined(__FAST_MATH__)
#error "the oracle must not be built with fast-math"
#endif

#define REAL float
#define SFX f32
#include "jdob_oracle_body.h"
#undef REAL
#undef SFX

#define REAL double
#define SFX f64
#include "jdob_oracle_body.h"
#undef REAL
#undef SFX
