// Host build of the library's E2M1 / E4M3 routines (the same header the GPU
// kernels include), exported for the CPU test that compares them with the
// oracle's independent implementation.
#include "formats.h"

extern "C" {
float host_e2m1_round(float y) { return quasar::e2m1_round(y); }
unsigned host_e2m1_code_of(float q) { return quasar::e2m1_code_of(q); }
double host_e4m3_round(double x, unsigned* code) { return quasar::e4m3_round(x, code); }
float host_e4m3_round_f32(float x, unsigned* code) { return quasar::e4m3_round_f32(x, code); }
}
