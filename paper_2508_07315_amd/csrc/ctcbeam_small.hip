// Instantiation unit: the small-beam decoder (K <= 8, V <= 1024, no boosting).
#include "ctcbeam_small.inl"
