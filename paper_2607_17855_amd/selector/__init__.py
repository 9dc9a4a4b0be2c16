"""Fitting of the kernel-family selector (csrc/selector.cpp) from timings."""
