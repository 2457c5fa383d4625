"""Plain CPU oracle of the brute-force device-mapping search (test infrastructure only)."""
