"""CPU oracle for the decoder step.  TEST INFRASTRUCTURE ONLY (see mtref.h)."""
