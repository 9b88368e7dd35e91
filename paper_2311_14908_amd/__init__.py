"""Kernel-SVM training (SMO, maximal violating pair) on one MI355X."""
