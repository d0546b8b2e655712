// Instantiations of the several-token kernel for general factor codes (ranks
// that are not multiples of 4, ARCHEAD_I5 core-left codes).
#define ARCHEAD_MID_GEN 1
#include "k_mid.hip"
