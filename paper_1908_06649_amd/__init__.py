"""MI355X (gfx950) implementation of the (m,l)-TCU hot path: the native
tall-left tensor-unit call and the blocked dense multiplication composed of
such calls (Section 3 model definition; Theorem 2 in Section 4.1)."""
