"""CPU oracle for the QK4PV8 attention path (test infrastructure only)."""
