"""CPU oracle (test infrastructure): full layer-wise recompute + structural affected sets."""
