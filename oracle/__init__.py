"""CPU oracle for the SRU layer: test infrastructure, never the product path."""
